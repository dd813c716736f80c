"""Pins of the oracle's channel scales: a ScaledArray whose scale is
broadcastable to its data (Section 2), here one power of two per row of A
(per output row) and one per column of B (per output column) on top of the
scalar scales, folded into the matmul's pre-cast value.

Each test fixes the rule by a route other than the oracle's own code: exact
rational sums of the decoded operands with the channel factors applied to
the inputs, the invariance of the true value under moving a power of two
between the scalar and the channel scale (the paper's model invariance), and
the reduction to the scalar path.
"""
from fractions import Fraction

import numpy as np
import pytest

from oracle import oracle as orc


def _codes(fmt, rng, shape, vmax=6):
    vals = rng.integers(-vmax, vmax + 1, shape).astype(np.float32)
    return orc.cast(fmt, vals)


def test_channel_scales_equal_scaling_the_decoded_inputs_exactly():
    """w * 2^e_w must equal sum_k (a_ik s_a c_i) (b_kj s_b d_j) computed with
    exact rationals from the decoded codes: the row factors follow the rows
    of A, the column factors the columns of B (swapping them, or negating an
    exponent, fails on this non-square case with distinct exponents)."""
    rng = np.random.default_rng(3)
    M, N, K = 5, 7, 24
    A = _codes(orc.E4M3, rng, (M, K))
    B = _codes(orc.E5M2, rng, (K, N))
    ea = rng.integers(-9, 10, M)
    eb = rng.integers(-9, 10, N)
    s_a, s_b = 2.0 ** -3, 2.0 ** 5
    acc = orc.matmul_acc(A, orc.E4M3, False, B, orc.E5M2, False).astype(np.float32)
    w, _, e_w, e_cc = orc.fused_pre(acc, s_a, s_b, K, ch_a=2.0 ** ea, ch_b=2.0 ** eb)
    assert e_cc == orc.matmul_scale_log2(K)
    dA, dB = orc.decode(orc.E4M3, A), orc.decode(orc.E5M2, B)
    for i in range(M):
        for j in range(N):
            exact = sum(Fraction(float(dA[i, k])) * Fraction(s_a) * Fraction(2) ** int(ea[i]) *
                        Fraction(float(dB[k, j])) * Fraction(s_b) * Fraction(2) ** int(eb[j])
                        for k in range(K))
            assert Fraction(float(w[i, j])) * Fraction(2) ** e_w == exact, (i, j)


@pytest.mark.parametrize("with_residual", [False, True])
@pytest.mark.parametrize("act", [orc.ACT_NONE, orc.ACT_RELU, orc.ACT_GELU_TANH])
def test_moving_a_power_of_two_between_scalar_and_channel_scale(with_residual, act):
    """A = A_d * s_a * c is the same tensor as A_d * (s_a 2^k) * (c 2^-k): the
    true pre-cast values and the final codes and scale must not change
    (Section 2's invariance of the represented value)."""
    rng = np.random.default_rng(11 + with_residual + 2 * act)
    M, N, K = 6, 9, 64
    acc = (rng.standard_normal((M, N)) * 20).astype(np.float32)
    ca = 2.0 ** rng.integers(-4, 5, M)
    cb = 2.0 ** rng.integers(-4, 5, N)
    res = None
    if with_residual:
        res = (orc.cast(orc.E4M3, rng.standard_normal((M, N)).astype(np.float32)), orc.E4M3, 2.0 ** 4)
    ref = orc.matmul_epilogue_fused(acc, 2.0 ** -2, 2.0 ** 3, K, res, act, ch_a=ca, ch_b=cb)
    w0, _, e0, _ = orc.fused_pre(acc, 2.0 ** -2, 2.0 ** 3, K, res, act, ca, cb)
    for k in (-3, 2, 5):
        got = orc.matmul_epilogue_fused(acc, 2.0 ** (-2 + k), 2.0 ** 3, K, res, act,
                                        ch_a=ca * 2.0 ** -k, ch_b=cb)
        assert np.array_equal(got[0], ref[0]) and got[1] == ref[1]
        w1, _, e1, _ = orc.fused_pre(acc, 2.0 ** -2, 2.0 ** (3 + k), K, res, act, ca, cb * 2.0 ** -k)
        # the same number wherever it is a normal fp32 in both scales (a
        # power-of-two shift commutes with the one rounding there)
        v0 = w0.astype(np.float64) * 2.0 ** e0
        v1 = w1.astype(np.float64) * 2.0 ** e1
        tiny = 2.0 ** (-126 + max(e0, e1))
        big = (np.abs(v0) >= tiny) & (np.abs(v1) >= tiny)
        assert np.array_equal(v1[big], v0[big])
        # every other value lies below the normal range of the coarser scale
        # on both sides: the far tail of a smooth gate, zero or subnormal
        assert np.all(np.abs(v0[~big]) < tiny) and np.all(np.abs(v1[~big]) < tiny)
        if act in (orc.ACT_NONE, orc.ACT_RELU):
            # no tail: relu's zeros (and exact zeros) fall in the same places
            assert np.array_equal(w1 == 0, w0 == 0)
            assert big.sum() == np.count_nonzero(w0)


def test_unit_channel_scales_reduce_to_the_scalar_path():
    rng = np.random.default_rng(21)
    M, N, K = 8, 5, 100
    acc = (rng.standard_normal((M, N)) * 7).astype(np.float32)
    res = (orc.cast(orc.E5M2, rng.standard_normal((1, N)).astype(np.float32)), orc.E5M2, 2.0)
    for r in (None, res):
        a = orc.fused_pre(acc, 0.5, 4.0, K, r, orc.ACT_SILU)
        b = orc.fused_pre(acc, 0.5, 4.0, K, r, orc.ACT_SILU, np.ones(M), np.ones(N))
        assert np.array_equal(a[0], b[0]) and a[2:] == b[2:]


def test_residual_with_channel_scales_on_an_integer_grid():
    """Integer accumulators, residual values and power-of-two factors keep
    every term exact: w * 2^e_w = acc s_a s_b c_i d_j + r s_r exactly."""
    rng = np.random.default_rng(8)
    M, N, K = 4, 6, 256
    acc = rng.integers(-500, 501, (M, N)).astype(np.float32)
    rv = rng.integers(-8, 9, (M, N)).astype(np.float32)
    codes = orc.cast(orc.F16, rv)
    ea, eb = rng.integers(-3, 4, M), rng.integers(-3, 4, N)
    w, _, e_w, e_cc = orc.fused_pre(acc, 2.0, 0.25, K, (codes, orc.F16, 2.0 ** 6), orc.ACT_NONE,
                                    2.0 ** ea, 2.0 ** eb)
    assert e_cc == 0 and e_w == max(1 - 2 + orc.matmul_scale_log2(K), 6)
    want = (acc.astype(np.float64) * 2.0 ** (1 - 2) * 2.0 ** ea[:, None] * 2.0 ** eb[None, :] +
            rv.astype(np.float64) * 2.0 ** 6)
    assert np.array_equal(w.astype(np.float64) * 2.0 ** e_w, want)


def test_channel_scale_must_be_a_power_of_two():
    acc = np.ones((2, 3), dtype=np.float32)
    with pytest.raises(ValueError):
        orc.fused_pre(acc, 1.0, 1.0, 4, ch_a=np.array([1.0, 3.0]))
    with pytest.raises(ValueError):
        orc.fused_pre(acc, 1.0, 1.0, 4, ch_b=np.array([1.0, 0.0, 2.0]))
