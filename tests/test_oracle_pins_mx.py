"""Pins of the oracle's MX block scales: a ScaledArray whose scale is
broadcastable to its data (Section 2), here one E8M0 byte (value
2^(byte - 127)) per 32 consecutive k of each row of A and of each column of
B, the block-scaling formats the section names, on top of the scalar scales.

Each test fixes the rule by a route other than the oracle's own loop:
exact rational sums over the decoded codes with the block factors applied
to the inputs, the reduction to the unscaled accumulator (all bytes 127)
and to per-channel factors (constant bytes along k), the decomposition of
the sum into its 32-k blocks, and the invariance under storage order.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import oracle as orc


def _codes(fmt, rng, shape, vmax=6.0):
    vals = (rng.standard_normal(shape) * vmax).astype(np.float32)
    return orc.cast(fmt, vals)


def _scales(rng, rows, K, lo=-12, hi=12, pad=None):
    ld = orc.mx_block_scale_ld(K)
    s = (127 + rng.integers(lo, hi + 1, (rows, ld))).astype(np.uint8)
    if pad is not None:
        s[:, (K + 31) // 32:] = pad
    return s


def _half_ulp_f32(x: float) -> Fraction:
    m, e = np.frexp(np.float32(x))
    e = max(int(e), -125)  # subnormal spacing below 2^-126
    return Fraction(2) ** (e - 24 - 1)


@pytest.mark.parametrize("fa,fb", [(orc.E4M3, orc.E4M3), (orc.E4M3, orc.E5M2), (orc.E5M2, orc.E5M2)])
def test_block_scales_are_the_exact_sum_of_scaled_inputs(fa, fb):
    """acc[i, j] is within half an fp32 ulp of sum_k a_ik 2^(sa[i, k//32]-127)
    b_kj 2^(sb[j, k//32]-127), computed with exact rationals; K = 70 has a
    partial third block, and the non-square shape with distinct bytes per
    row, column and block separates rows from columns and k // 32 from
    other block maps."""
    rng = np.random.default_rng(5 + fa + 2 * fb)
    M, N, K = 4, 3, 70
    A = _codes(fa, rng, (M, K))
    B = _codes(fb, rng, (K, N))
    sa = _scales(rng, M, K)
    sb = _scales(rng, N, K)
    acc = orc.matmul_acc_mx(A, fa, False, B, fb, False, sa, sb)
    dA, dB = orc.decode(fa, A), orc.decode(fb, B)
    for i in range(M):
        for j in range(N):
            exact = sum(Fraction(float(dA[i, k])) * Fraction(2) ** (int(sa[i, k // 32]) - 127) *
                        Fraction(float(dB[k, j])) * Fraction(2) ** (int(sb[j, k // 32]) - 127)
                        for k in range(K))
            got = Fraction(float(acc[i, j]))
            assert abs(got - exact) <= _half_ulp_f32(float(acc[i, j])), (i, j, float(exact))


def test_unit_block_scales_reduce_to_the_plain_accumulator():
    rng = np.random.default_rng(21)
    M, N, K = 9, 11, 200
    A = _codes(orc.E4M3, rng, (M, K))
    B = _codes(orc.E5M2, rng, (K, N))
    ld = orc.mx_block_scale_ld(K)
    one_a = np.full((M, ld), 127, np.uint8)
    one_b = np.full((N, ld), 127, np.uint8)
    got = orc.matmul_acc_mx(A, orc.E4M3, False, B, orc.E5M2, False, one_a, one_b)
    ref = orc.matmul_acc(A, orc.E4M3, False, B, orc.E5M2, False)
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))


def test_constant_bytes_along_k_are_channel_factors():
    """Bytes constant along k act as one power of two per row of A and per
    column of B: the accumulator is the plain one times 2^(ca_i + cb_j),
    exactly (a power-of-two product inside fp32's normal range)."""
    rng = np.random.default_rng(22)
    M, N, K = 6, 10, 160
    A = _codes(orc.E4M3, rng, (M, K))
    B = _codes(orc.E4M3, rng, (K, N))
    ca = rng.integers(-20, 21, M)
    cb = rng.integers(-20, 21, N)
    ld = orc.mx_block_scale_ld(K)
    sa = np.repeat((127 + ca)[:, None], ld, axis=1).astype(np.uint8)
    sb = np.repeat((127 + cb)[:, None], ld, axis=1).astype(np.uint8)
    got = orc.matmul_acc_mx(A, orc.E4M3, False, B, orc.E4M3, False, sa, sb)
    ref = orc.matmul_acc(A, orc.E4M3, False, B, orc.E4M3, False).astype(np.float64)
    want = (ref * np.exp2(ca[:, None] + cb[None, :])).astype(np.float32)
    assert np.array_equal(got, want)


def test_sum_splits_into_its_32k_blocks():
    """acc equals sum over blocks b of 2^(sa[i,b]+sb[j,b]-254) times the
    plain accumulator of the k-slice [32 b, 32 b + 32): the byte of column
    k // 32 scales exactly the k of that slice. Integer-valued codes keep
    every block sum exact, so the comparison is exact."""
    rng = np.random.default_rng(23)
    M, N, K = 5, 7, 32 * 5 + 9
    A = orc.cast(orc.E4M3, rng.integers(-8, 9, (M, K)).astype(np.float32))
    B = orc.cast(orc.E4M3, rng.integers(-8, 9, (K, N)).astype(np.float32))
    sa = _scales(rng, M, K, -6, 6)
    sb = _scales(rng, N, K, -6, 6)
    got = orc.matmul_acc_mx(A, orc.E4M3, False, B, orc.E4M3, False, sa, sb)
    want = np.zeros((M, N))
    for b in range((K + 31) // 32):
        k0, k1 = 32 * b, min(K, 32 * b + 32)
        part = orc.matmul_acc(A[:, k0:k1], orc.E4M3, False, B[k0:k1], orc.E4M3, False).astype(np.float64)
        want += part * np.exp2(sa[:, b].astype(np.int64)[:, None] + sb[:, b].astype(np.int64)[None, :] - 254)
    assert np.array_equal(got, want.astype(np.float32))


def test_padding_bytes_are_never_read_and_nan_bytes_are_rejected():
    rng = np.random.default_rng(24)
    M, N, K = 3, 4, 70  # 3 blocks used of the 4 in a row
    A = _codes(orc.E4M3, rng, (M, K))
    B = _codes(orc.E4M3, rng, (K, N))
    sa = _scales(rng, M, K, pad=127)
    sb = _scales(rng, N, K, pad=127)
    ref = orc.matmul_acc_mx(A, orc.E4M3, False, B, orc.E4M3, False, sa, sb)
    sa2, sb2 = sa.copy(), sb.copy()
    sa2[:, 3] = 0xFF
    sb2[:, 3] = 0
    got = orc.matmul_acc_mx(A, orc.E4M3, False, B, orc.E4M3, False, sa2, sb2)
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))
    sa2[1, 2] = 0xFF
    with pytest.raises(ValueError):
        orc.matmul_acc_mx(A, orc.E4M3, False, B, orc.E4M3, False, sa2, sb)


def test_storage_order_and_sampled_positions_agree():
    rng = np.random.default_rng(25)
    M, N, K = 7, 5, 100
    A = _codes(orc.E5M2, rng, (M, K))
    B = _codes(orc.E4M3, rng, (K, N))
    sa = _scales(rng, M, K)
    sb = _scales(rng, N, K)
    ref = orc.matmul_acc_mx(A, orc.E5M2, False, B, orc.E4M3, False, sa, sb)
    for ta in (False, True):
        for tb in (False, True):
            A_st = A.T.copy() if ta else A
            B_st = B.T.copy() if tb else B
            got = orc.matmul_acc_mx(A_st, orc.E5M2, ta, B_st, orc.E4M3, tb, sa, sb)
            assert np.array_equal(got.view(np.uint32), ref.view(np.uint32)), (ta, tb)
    ii, jj = np.array([0, 6, 3]), np.array([4, 0, 2])
    at, l1 = orc.matmul_acc_mx_at(A, orc.E5M2, False, B, orc.E4M3, False, sa, sb, ii, jj)
    assert np.array_equal(at, ref[ii, jj])
    absA, absB = A & 0x7F, B & 0x7F  # sign-magnitude codes: |value|
    l1_ref = orc.matmul_acc_mx(absA, orc.E5M2, False, absB, orc.E4M3, False, sa, sb)
    assert np.allclose(l1, l1_ref[ii, jj], rtol=1e-6)


def test_mx_golden_subnormal_accumulator():
    """Hand-derived (tests/golden/epilogue_examples.json): block scales can
    make the accumulator an fp32 subnormal; the block-scaled sum keeps it
    exactly and the epilogue casts it with one power-of-two shift."""
    path = os.path.join(os.path.dirname(__file__), "golden", "epilogue_examples.json")
    with open(path) as f:
        cases = json.load(f)["mx_cases"]
    for c in cases:
        A = np.array(c["a_codes"], dtype=np.uint8)
        B = np.array(c["b_codes"], dtype=np.uint8)
        K = A.shape[1]
        acc = orc.matmul_acc_mx(A, orc.E4M3, False, B, orc.E4M3, False,
                                np.array(c["a_block"], np.uint8), np.array(c["b_block"], np.uint8))
        want = [[math.ldexp(v[0], v[1]) for v in row] for row in c["acc"]]
        assert acc.tolist() == want, c["name"]
        codes, e_out, _ = orc.matmul_epilogue(acc, 2.0 ** c["a_scale_log2"],
                                              2.0 ** c["b_scale_log2"], K, orc.RESCALE_AMAX)
        assert codes.tolist() == c["out_codes"] and e_out == c["out_scale_log2"], c["name"]
