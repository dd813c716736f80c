"""Pins of the oracle's fused scaled add and activation (the matmul epilogue
extension of Algorithm 3's add rule and Appendix C.1's activation rule).

Each test fixes one part by a route other than the oracle's own code: closed
forms (the power-of-two add rule, sigmoid symmetry), an independent library
routine (math.erf for the exact GELU the tanh form approximates), exact
rational or integer arithmetic, hand-derived examples (tests/golden/) and
the model invariance the paper states for a scaled activation.
"""
import json
import math
import os

import numpy as np
import pytest

from oracle import oracle as orc

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
FMT = {"e4m3": orc.E4M3, "e5m2": orc.E5M2, "f16": orc.F16}
ACT = {"none": orc.ACT_NONE, "relu": orc.ACT_RELU, "gelu": orc.ACT_GELU_TANH, "silu": orc.ACT_SILU}
MODE = {"none": orc.RESCALE_NONE, "amax": orc.RESCALE_AMAX}


# ----------------------------------------------------------------------------- gates

@pytest.mark.parametrize("act", [orc.ACT_GELU_TANH, orc.ACT_SILU])
def test_smooth_gates_are_sigmoids_of_odd_functions(act):
    """g(x) + g(-x) = 1 and g(0) = 1/2: both gates are a sigmoid (tanh form:
    (1 + tanh(u))/2) of an odd function of x, so f(x) - f(-x) = x. A sign
    slip in the exponent or in the cubic term breaks the symmetry."""
    xs = np.linspace(-12.0, 12.0, 481)
    for x in xs:
        assert abs(orc.gate(act, x) + orc.gate(act, -x) - 1.0) < 4e-16
    assert orc.gate(act, 0.0) == 0.5
    # monotone from 0 to 1
    g = np.array([orc.gate(act, x) for x in xs])
    assert np.all(np.diff(g) >= 0) and g[0] < 1e-5 and g[-1] > 1 - 1e-5


def test_silu_gate_closed_form_points():
    """sigmoid(ln 3) = 3/4, sigmoid(-ln 3) = 1/4, sigmoid(ln 7) = 7/8."""
    assert abs(orc.gate(orc.ACT_SILU, math.log(3.0)) - 0.75) < 1e-15
    assert abs(orc.gate(orc.ACT_SILU, -math.log(3.0)) - 0.25) < 1e-15
    assert abs(orc.gate(orc.ACT_SILU, math.log(7.0)) - 0.875) < 1e-15


def test_gelu_tanh_form_approximates_the_exact_gelu_to_its_known_error():
    """The tanh form approximates x * Phi(x) (Phi from math.erf, an independent
    routine) with a maximum error of about 4.73e-4 near |x| = 2.7. A wrong
    constant (sqrt(2/pi) or 0.044715) moves that maximum outside the band."""
    xs = np.linspace(-10.0, 10.0, 200001)
    err = max(abs(x * orc.gate(orc.ACT_GELU_TANH, x) - 0.5 * x * (1.0 + math.erf(x / math.sqrt(2.0))))
              for x in xs[::7])
    assert 4.6e-4 < err < 4.8e-4


@pytest.mark.parametrize("act", [orc.ACT_GELU_TANH, orc.ACT_SILU])
def test_smooth_gates_keep_their_digits_in_the_negative_tail(act):
    """Against 60-digit decimal arithmetic (an independent evaluation of
    (1 + tanh(u))/2 = e^u / (e^u + e^-u), and of 1 / (1 + e^-x)): fp64
    relative accuracy (1e-13, the rounding of the argument amplified by
    |2u| < 150) down to gates of 1e-30, where the naive 1 + tanh(u) would
    have cancelled to 0."""
    from decimal import Decimal, getcontext
    getcontext().prec = 60
    k = Decimal(2) / Decimal("3.14159265358979323846264338327950288419716939937510582097494")
    k = k.sqrt()
    for x in np.linspace(-12.0, 2.0, 141):
        d = Decimal(float(x))
        if act == orc.ACT_GELU_TANH:
            u = k * (d + Decimal("0.044715") * d * d * d)
            ref = u.exp() / (u.exp() + (-u).exp())
        else:
            ref = 1 / (1 + (-d).exp())
        if ref < Decimal("1e-30"):
            continue
        got = Decimal(orc.gate(act, float(x)))
        assert abs(got - ref) <= ref * Decimal("1e-13"), (x, got, ref)


def test_relu_gate_is_the_step():
    for x in [1e-300, 0.5, 3.0, 1e300, float("inf")]:
        assert orc.gate(orc.ACT_RELU, x) == 1.0
    for x in [0.0, -0.0, -1e-300, -2.0, float("-inf")]:
        assert orc.gate(orc.ACT_RELU, x) == 0.0


@pytest.mark.parametrize("act", [orc.ACT_GELU_TANH, orc.ACT_SILU])
def test_gate_limits_at_infinity(act):
    """g is defined at +-inf (1 and 0), the property Appendix C.1 relies on
    when X_d * X_s overflows."""
    assert orc.gate(act, float("inf")) == 1.0
    assert orc.gate(act, float("-inf")) == 0.0
    assert math.isnan(orc.gate(act, float("nan")))


# ----------------------------------------------------------------------------- add rule

def test_add_scale_rule_is_the_larger_scale():
    """sqrt(4^a + 4^b) lies in [2^max(a,b), 2^(max(a,b)+1/2)], so rounding it
    down to a power of two gives the larger of the two scales."""
    for a in range(-60, 61, 3):
        for b in range(-60, 61, 7):
            assert orc.add_scale_log2(a, b) == max(a, b), (a, b)


def _small_int_codes(fmt, rng, shape):
    """Codes whose decoded values are integers in [-8, 8]."""
    vals = rng.integers(-8, 9, shape).astype(np.float32)
    return orc.cast(fmt, vals), vals.astype(np.float64)


@pytest.mark.parametrize("res_fmt", [orc.E4M3, orc.E5M2, orc.F16])
@pytest.mark.parametrize("broadcast", [False, True])
def test_scaled_add_is_exact_on_an_integer_grid(res_fmt, broadcast):
    """With integer accumulators and residual values and power-of-two scales
    the sum is exact in fp32: the true value w * 2^e_w must equal
    acc * s_a * s_b + r * s_r exactly (a wrong shift of either term, or the
    wrong residual row, fails)."""
    rng = np.random.default_rng(5 + res_fmt + 10 * broadcast)
    M, N, K = 7, 11, 300
    acc = rng.integers(-3000, 3001, (M, N)).astype(np.float32)
    codes, r = _small_int_codes(res_fmt, rng, (1 if broadcast else M, N))
    for e_a, e_b, q in [(0, 0, 0), (-3, 2, 9), (4, 1, -6), (2, 2, 6)]:
        w, y64, e_w, e_cc = orc.fused_pre(acc, 2.0 ** e_a, 2.0 ** e_b, K, (codes, res_fmt, 2.0 ** q))
        assert e_cc == 0
        assert e_w == max(e_a + e_b + orc.matmul_scale_log2(K), q)
        want = acc.astype(np.float64) * 2.0 ** (e_a + e_b) + np.broadcast_to(r, (M, N)) * 2.0 ** q
        assert np.array_equal(w.astype(np.float64) * 2.0 ** e_w, want)
        assert np.array_equal(y64, w.astype(np.float64))


def test_hand_examples():
    """tests/golden/fused_examples.json: hand-derived add / relu / bias cases."""
    with open(os.path.join(GOLDEN, "fused_examples.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        acc = np.array(c["acc"], dtype=np.float32).reshape(c["M"], c["N"])
        res = None
        if c["residual"] is not None:
            rr = c["residual"]
            dt = np.uint16 if rr["fmt"] == "f16" else np.uint8
            codes = np.array(rr["codes"], dtype=dt).reshape(rr["rows"], c["N"])
            res = (codes, FMT[rr["fmt"]], 2.0 ** rr["scale_log2"])
        out, e_out, amax, w, _ = orc.matmul_epilogue_fused(
            acc, 2.0 ** c["a_scale_log2"], 2.0 ** c["b_scale_log2"], c["K"], res, ACT[c["act"]],
            MODE[c["mode"]], out_fmt=FMT[c["out_fmt"]])
        assert w.ravel().tolist() == c["w"], c["name"]
        assert np.array_equal(np.signbit(w.ravel()), np.signbit(np.array(c["w"]))), c["name"]
        assert out.ravel().tolist() == c["out_codes"], c["name"]
        assert e_out == c["out_scale_log2"], c["name"]
        assert amax == c["amax"], c["name"]
        _, _, e_w, _ = orc.fused_pre(acc, 2.0 ** c["a_scale_log2"], 2.0 ** c["b_scale_log2"], c["K"],
                                     res, ACT[c["act"]])
        assert e_w == c["e_w"], c["name"]


# ----------------------------------------------------------------------------- activation rule

@pytest.mark.parametrize("act", [orc.ACT_RELU, orc.ACT_GELU_TANH, orc.ACT_SILU])
def test_scaled_activation_equals_the_unscaled_one(act):
    """Appendix C.1: f_scaled(X_d, X_s) = (X_d * g(X_d * X_s), X_s) represents
    f(X) for X = X_d * X_s. So the fused output at scales (2^e_a, 2^e_b) must
    decode to f of the true product value: the gate sees the scaled value, not
    the data (gelu and silu are not scale-invariant, so evaluating g at X_d
    fails)."""
    rng = np.random.default_rng(17 + act)
    acc = (rng.standard_normal((20, 30)) * 3.0).astype(np.float32)
    for e_a, e_b in [(0, 0), (3, -1), (-4, -2), (5, 2)]:
        w, y64, e_w, e_cc = orc.fused_pre(acc, 2.0 ** e_a, 2.0 ** e_b, 64, None, act)
        assert e_w == e_a + e_b and e_cc == orc.matmul_scale_log2(64)
        x = acc.astype(np.float64) * 2.0 ** (e_a + e_b)
        fx = np.array([xi * orc.gate(act, xi) for xi in x.ravel()]).reshape(x.shape)
        got = y64 * 2.0 ** e_w
        assert np.allclose(got, fx, rtol=1e-15, atol=0)
        assert np.array_equal(w, y64.astype(np.float32))
    if act != orc.ACT_RELU:
        # the same data at another scale gives another function of the data
        w0 = orc.fused_pre(acc, 1.0, 1.0, 64, None, act)[0]
        w1 = orc.fused_pre(acc, 2.0 ** 3, 1.0, 64, None, act)[0]
        assert not np.array_equal(w0, w1)


def test_relu_keeps_positives_and_zeroes_the_rest():
    acc = np.array([[3.5, -2.0, 0.0, -0.0, 1e-30, -1e30, np.inf, -np.inf, np.nan]], dtype=np.float32)
    w, _, _, _ = orc.fused_pre(acc, 1.0, 1.0, 1, None, orc.ACT_RELU)
    assert w[0, 0] == 3.5 and w[0, 4] == np.float32(1e-30) and w[0, 6] == np.inf
    assert np.all(w[0, [1, 2, 3, 5]] == 0.0)
    # f(x) = x * g(x): -inf * 0 and NaN * g are NaN
    assert np.isnan(w[0, 7]) and np.isnan(w[0, 8])


@pytest.mark.parametrize("act", [orc.ACT_GELU_TANH, orc.ACT_SILU])
def test_gate_at_an_overflowing_scaled_value(act):
    """X_d * X_s beyond the fp32 range: the gate is still defined (Appendix
    C.1), so the output is X_d (x > 0) or 0 (x < 0) times the scale."""
    acc = np.array([[1.5, -1.5, 3.0]], dtype=np.float32)
    w, _, e_w, _ = orc.fused_pre(acc, 2.0 ** 100, 2.0 ** 100, 1, None, act)
    assert e_w == 200
    assert w[0, 0] == 1.5 and w[0, 2] == 3.0
    assert w[0, 1] == 0.0


# ----------------------------------------------------------------------------- composition

@pytest.mark.parametrize("out_fmt", [orc.E4M3, orc.E5M2, orc.F16])
@pytest.mark.parametrize("mode", [orc.RESCALE_NONE, orc.RESCALE_AMAX])
@pytest.mark.parametrize("target", [0, 4])
def test_no_add_no_activation_is_the_plain_epilogue(out_fmt, mode, target):
    """The fused epilogue with nothing fused reduces to the pinned matmul
    epilogue (same codes, output scale and statistic), and its delayed form
    to the pinned delayed epilogue."""
    rng = np.random.default_rng(3 + out_fmt + 3 * mode + target)
    acc = (rng.standard_normal((33, 17)) * 2.0 ** rng.integers(-10, 12, (33, 17))).astype(np.float32)
    acc[0, 0] = np.nan
    acc[1, 1] = -0.0
    for s_a, s_b, K in [(1.0, 1.0, 1), (2.0 ** -3, 2.0 ** 6, 5000), (2.0 ** 7, 2.0 ** 1, 37)]:
        ref = orc.matmul_epilogue(acc, s_a, s_b, K, mode, target, True, out_fmt)
        got = orc.matmul_epilogue_fused(acc, s_a, s_b, K, None, orc.ACT_NONE, mode, target,
                                        out_fmt=out_fmt)
        assert np.array_equal(ref[0], got[0]) and ref[1] == got[1] and ref[2] == got[2]
        for stat in [0.0, 3.0, 2.0 ** -7, float("nan")]:
            ref = orc.matmul_epilogue_delayed(acc, s_a, s_b, K, stat, target, True, out_fmt)
            got = orc.matmul_epilogue_fused(acc, s_a, s_b, K, None, orc.ACT_NONE,
                                            orc.RESCALE_DELAYED, target, stat, True, out_fmt)
            assert np.array_equal(ref[0], got[0]) and ref[1] == got[1] and ref[2] == got[2]


def test_rescale_statistic_is_over_the_activated_values():
    """The amax rescale after a fused relu measures the relu output: with the
    largest magnitude negative, the statistic is the largest positive one."""
    acc = np.array([[-100.0, 3.0, 5.0, -7.0]], dtype=np.float32)
    _, e_out, amax, _, _ = orc.matmul_epilogue_fused(acc, 1.0, 1.0, 1, None, orc.ACT_RELU,
                                                     orc.RESCALE_AMAX)
    assert amax == 5.0 and e_out == 2
    _, e_out, amax, _, _ = orc.matmul_epilogue_fused(acc, 1.0, 1.0, 1, None, orc.ACT_NONE,
                                                     orc.RESCALE_AMAX)
    assert amax == 100.0 and e_out == 6


def test_residual_specials_propagate():
    """An Inf residual makes the sum Inf (amax Inf: no rebalance, saturating
    cast to the max code); a NaN residual gives NaN, which the statistic
    skips and the cast keeps."""
    acc = np.array([[1.0, 2.0, 3.0]], dtype=np.float32)
    res = np.array([[0x7C, 0x7D, 0x3C]], dtype=np.uint8)        # E5M2 +Inf, NaN, 1.0
    out, e_out, amax, w, _ = orc.matmul_epilogue_fused(acc, 1.0, 1.0, 1, (res, orc.E5M2, 1.0),
                                                       orc.ACT_NONE, orc.RESCALE_AMAX)
    assert w[0, 0] == np.inf and np.isnan(w[0, 1]) and w[0, 2] == 4.0
    assert amax == np.inf and e_out == 0
    assert out[0, 0] == 0x7E and out[0, 1] == 0x7F and out[0, 2] == 0x48


def test_fused_matches_exact_rational_arithmetic_on_tiny_cases():
    """Brute force with fractions: relu(A @ B * s_a * s_b + R * s_r) for tiny
    integer-valued inputs, against the decoded fused output times its scale,
    within half a code of the output format (E4M3 relative 2^-4)."""
    from fractions import Fraction
    rng = np.random.default_rng(23)
    for trial in range(20):
        M, N, K = 3, 4, int(rng.integers(1, 6))
        A = rng.integers(-4, 5, (M, K)).astype(np.float32)
        B = rng.integers(-4, 5, (K, N)).astype(np.float32)
        R = rng.integers(-6, 7, (M, N)).astype(np.float32)
        e_a, e_b, q = (int(v) for v in rng.integers(-3, 4, 3))
        acc = (A.astype(np.float64) @ B.astype(np.float64)).astype(np.float32)
        rc = orc.cast(orc.E4M3, R)
        out, e_out, _, _, _ = orc.matmul_epilogue_fused(acc, 2.0 ** e_a, 2.0 ** e_b, K,
                                                        (rc, orc.E4M3, 2.0 ** q), orc.ACT_RELU,
                                                        orc.RESCALE_AMAX)
        got = orc.decode(orc.E4M3, out) * 2.0 ** e_out
        for i in range(M):
            for j in range(N):
                s = sum(Fraction(int(A[i, k])) * int(B[k, j]) for k in range(K))
                v = s * Fraction(2) ** (e_a + e_b) + Fraction(int(R[i, j])) * Fraction(2) ** q
                v = v if v > 0 else Fraction(0)
                assert abs(Fraction(got[i, j]) - v) <= abs(v) / 16, (trial, i, j)
