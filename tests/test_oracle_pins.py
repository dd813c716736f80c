"""Pins of the CPU oracle against things other than itself.

Each test fixes one part of the oracle by a route that does not go through
the oracle's own code: a library routine (torch / numpy float8 and float16
conversions), a closed form, exact rational arithmetic, integer arithmetic,
hand-derived worked examples (tests/golden/), or an invariant the paper
states (model invariance, Section 1; lossless power-of-two rescale,
Section 2). The paper prints no numeric worked example for this path.
"""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import oracle as orc

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

TORCH_F8 = {orc.E4M3: torch.float8_e4m3fn, orc.E5M2: torch.float8_e5m2}


def torch_decode8(fmt, codes):
    t = torch.from_numpy(np.asarray(codes, dtype=np.uint8)).view(TORCH_F8[fmt])
    return t.to(torch.float64).numpy()


def same_or_both_nan(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return np.array_equal(np.isnan(a), np.isnan(b)) and np.array_equal(a[~np.isnan(a)], b[~np.isnan(b)]) \
        and np.array_equal(np.signbit(a[~np.isnan(a)]), np.signbit(b[~np.isnan(b)]))


# ----------------------------------------------------------------------------- decode

@pytest.mark.parametrize("fmt", [orc.E4M3, orc.E5M2])
def test_decode_all_fp8_codes_match_torch(fmt):
    codes = np.arange(256)
    assert same_or_both_nan(orc.decode(fmt, codes), torch_decode8(fmt, codes))


def test_decode_all_f16_codes_match_numpy():
    codes = np.arange(65536, dtype=np.uint32)
    ref = codes.astype(np.uint16).view(np.float16).astype(np.float64)
    assert same_or_both_nan(orc.decode(orc.F16, codes), ref)


def test_decode_landmarks_closed_form():
    d = lambda f, c: orc.decode(f, np.array([c]))[0]
    # OCP E4M3: max 448 = 1.75 * 2^8, min normal 2^-6, min subnormal 2^-9, NaN only S.1111.111
    assert d(orc.E4M3, 0x7E) == 448.0 and d(orc.E4M3, 0xFE) == -448.0
    assert d(orc.E4M3, 0x08) == 2.0 ** -6 and d(orc.E4M3, 0x01) == 2.0 ** -9
    nan_codes = [c for c in range(256) if math.isnan(d(orc.E4M3, c))]
    assert nan_codes == [0x7F, 0xFF]
    # OCP E5M2: max 57344 = 1.75 * 2^15, Inf at 0x7C, three NaN codes per sign
    assert d(orc.E5M2, 0x7B) == 57344.0 and d(orc.E5M2, 0x7C) == math.inf
    assert d(orc.E5M2, 0x01) == 2.0 ** -16 and d(orc.E5M2, 0x04) == 2.0 ** -14
    assert [c for c in range(128) if math.isnan(d(orc.E5M2, c))] == [0x7D, 0x7E, 0x7F]
    assert d(orc.E4M3, 0x80) == 0.0 and math.copysign(1, d(orc.E4M3, 0x80)) == -1


# ----------------------------------------------------------------------------- cast

def _structured_f32(exp_lo, exp_hi, top_bits, low_patterns):
    """All fp32 with biased exponent in [exp_lo, exp_hi], every value of the top
    `top_bits` mantissa bits, and the remaining bits drawn from low_patterns."""
    low_n = 23 - top_bits
    exps = np.arange(exp_lo, exp_hi + 1, dtype=np.uint32)
    tops = np.arange(1 << top_bits, dtype=np.uint32)
    lows = np.array(low_patterns, dtype=np.uint32) & ((1 << low_n) - 1)
    e, t, l = np.meshgrid(exps, tops, lows, indexing="ij")
    bits = (e << 23) | (t << low_n) | l
    bits = bits.ravel()
    bits = np.concatenate([bits, bits | np.uint32(0x80000000)])
    return bits.view(np.float32)


def _patterns(n_low):
    full = (1 << n_low) - 1
    half = 1 << (n_low - 1)
    return [0, 1, 2, half - 1, half, half + 1, full - 1, full]


@pytest.mark.parametrize("fmt", [orc.E4M3, orc.E5M2])
def test_cast_matches_torch_rne_in_and_out_of_range(fmt):
    # exponents 2^-30 .. 2^18: covers zero-rounding, subnormals, normals, overflow
    x = _structured_f32(127 - 30, 127 + 18, 9, _patterns(14))
    ours = orc.cast(fmt, x, saturate=False)
    ref = torch.from_numpy(x).to(TORCH_F8[fmt]).view(torch.uint8).numpy()
    assert np.array_equal(ours, ref), np.flatnonzero(ours != ref)[:10]


def test_cast_f16_matches_torch_rne():
    x = _structured_f32(127 - 27, 127 + 17, 11, _patterns(12))
    ours = orc.cast(orc.F16, x, saturate=False)
    ref = torch.from_numpy(x).to(torch.float16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_cast_random_matches_torch():
    rng = np.random.default_rng(7)
    bits = rng.integers(0, 2 ** 32, size=2_000_000, dtype=np.uint64).astype(np.uint32)
    x = bits.view(np.float32)
    x = x[~np.isnan(x)]
    for fmt in (orc.E4M3, orc.E5M2):
        ref = torch.from_numpy(x).to(TORCH_F8[fmt]).view(torch.uint8).numpy()
        assert np.array_equal(orc.cast(fmt, x, saturate=False), ref)
    ref16 = torch.from_numpy(x).to(torch.float16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(orc.cast(orc.F16, x, saturate=False), ref16)


def test_cast_saturation_and_specials_closed_form():
    c = lambda f, v, s: int(orc.cast(f, np.array([v], np.float32), saturate=s)[0])
    inf, nan = float("inf"), float("nan")
    # E4M3: 464 is the midpoint of 448 and the (virtual) 480; even code 0x7E wins
    assert c(orc.E4M3, 464.0, True) == 0x7E and c(orc.E4M3, 464.0, False) == 0x7E
    assert c(orc.E4M3, 464.0001, True) == 0x7E and c(orc.E4M3, 464.0001, False) == 0x7F
    assert c(orc.E4M3, 1e30, True) == 0x7E and c(orc.E4M3, -1e30, True) == 0xFE
    assert c(orc.E4M3, inf, True) == 0x7E and c(orc.E4M3, -inf, True) == 0xFE
    assert c(orc.E4M3, inf, False) == 0x7F and c(orc.E4M3, -inf, False) == 0xFF
    assert c(orc.E4M3, nan, True) == 0x7F and c(orc.E4M3, -nan, True) == 0xFF
    # E5M2: 61440 is the midpoint of 57344 and 65536 (code 0x7C even) -> overflow
    assert c(orc.E5M2, 61440.0, True) == 0x7B and c(orc.E5M2, 61440.0, False) == 0x7C
    assert c(orc.E5M2, 61439.996, False) == 0x7B
    assert c(orc.E5M2, inf, True) == 0x7B and c(orc.E5M2, -inf, False) == 0xFC
    # FP16: 65520 is the midpoint of 65504 and 65536 -> overflow
    assert c(orc.F16, 65520.0, True) == 0x7BFF and c(orc.F16, 65520.0, False) == 0x7C00
    assert c(orc.F16, 65519.996, False) == 0x7BFF
    assert c(orc.F16, nan, True) == 0x7E00
    # zeros and the subnormal tie at half the smallest subnormal (ties to 0, even)
    assert c(orc.E4M3, -0.0, True) == 0x80
    assert c(orc.E4M3, 2.0 ** -10, True) == 0x00
    assert c(orc.E4M3, 1.5 * 2.0 ** -9, True) == 0x02     # tie between codes 1 and 2 -> 2
    assert c(orc.E5M2, 2.0 ** -17, True) == 0x00
    assert c(orc.E5M2, 3 * 2.0 ** -17, True) == 0x02


def _fraction_nearest(fmt, x):
    """Brute force: nearest representable value by exact rational distance,
    ties to the even code; overflow beyond the midpoint to the next binade
    step saturates (the saturating reading)."""
    vals = []
    for code in range(128):
        v = orc.decode(fmt, np.array([code]))[0]
        if math.isfinite(v):
            vals.append((Fraction(v), code))
    top, below = vals[-1][0], vals[-2][0]
    ax = Fraction(abs(float(x)))
    best = None
    for v, code in vals + [(top + (top - below), vals[-1][1] + 1)]:
        dist = abs(ax - v)
        if best is None or dist < best[0] or (dist == best[0] and code % 2 == 0):
            best = (dist, code)
    code = min(best[1], vals[-1][1])
    return code | (0x80 if math.copysign(1.0, float(x)) < 0 else 0)


@pytest.mark.parametrize("fmt", [orc.E4M3, orc.E5M2])
def test_cast_matches_brute_force_fraction_search(fmt):
    rng = np.random.default_rng(11 + fmt)
    x = np.concatenate([
        rng.standard_normal(1500) * np.exp2(rng.uniform(-20, 17, 1500)),
        (np.arange(-64, 64) * 2.0 ** -11),            # dense subnormal ladder with ties
    ]).astype(np.float32)
    ours = orc.cast(fmt, x, saturate=True)
    ref = np.array([_fraction_nearest(fmt, v) for v in x], dtype=np.uint8)
    assert np.array_equal(ours, ref)


# ----------------------------------------------------------------------------- scale rule

def test_matmul_scale_rule_closed_form():
    # largest e with 2^e <= sqrt(K), from the integer square root
    for K in list(range(1, 5000)) + [8192, 11008, 12288, 16384, 2 ** 20 - 1, 2 ** 20, 2 ** 24]:
        r = math.isqrt(K)
        assert orc.matmul_scale_log2(K) == r.bit_length() - 1
    assert [orc.matmul_scale_log2(k) for k in (256, 2048, 4096, 8192, 11008, 12288, 16384)] == \
        [4, 5, 6, 6, 6, 6, 7]


def test_floor_log2_matches_frexp_on_fp32_grid():
    rng = np.random.default_rng(3)
    bits = rng.integers(1, 0x7F800000, size=200_000, dtype=np.int64).astype(np.uint32)
    x = bits.view(np.float32).astype(np.float64)
    ours = np.array([orc.floor_log2(v) for v in x[:20000]])
    ref = np.floor(np.log2(x[:20000])).astype(np.int64)
    # log2 of an exact power of two is exact in fp64, and no fp32 value lies
    # close enough to a power of two from below for floor(log2) to be misrounded
    assert np.array_equal(ours, ref)


# ----------------------------------------------------------------------------- accumulate

PAIRS = [(orc.E4M3, orc.E4M3), (orc.E4M3, orc.E5M2), (orc.E5M2, orc.E4M3), (orc.E5M2, orc.E5M2)]


@pytest.mark.parametrize("fa,fb", PAIRS)
def test_acc_all_code_pairs_outer_product(fa, fb):
    """Every one of the 65,536 code pairs, as a K=1 outer product, equals the
    fp64 product of torch-decoded values rounded to fp32."""
    A = np.arange(256, dtype=np.uint8).reshape(256, 1)
    B = np.arange(256, dtype=np.uint8).reshape(1, 256)
    acc = orc.matmul_acc(A, fa, False, B, fb, False)
    # the fp32 accumulator starts at +0, so an all-zero sum is +0
    ref = np.outer(torch_decode8(fa, np.arange(256)), torch_decode8(fb, np.arange(256))) + 0.0
    with np.errstate(invalid="ignore", over="ignore"):
        ref32 = ref.astype(np.float32)
    assert same_or_both_nan(acc, ref32)
    # zero-padding K leaves the sums unchanged (0 * finite adds +-0)
    A2 = np.concatenate([A, np.zeros((256, 3), np.uint8)], axis=1)
    B2 = np.concatenate([B, np.zeros((3, 256), np.uint8)], axis=0)
    acc2 = orc.matmul_acc(A2, fa, False, B2, fb, False)
    fin = np.isfinite(acc)
    assert np.array_equal(acc2[fin], acc[fin])


def _finite_codes(fmt, rng, n, exp_lo, exp_hi):
    out = []
    while len(out) < n:
        c = int(rng.integers(0, 256))
        v = orc.decode(fmt, np.array([c]))[0]
        if not math.isfinite(v):
            continue
        if v != 0 and not (exp_lo <= math.frexp(abs(v))[1] - 1 <= exp_hi):
            continue
        out.append(c)
    return np.array(out, dtype=np.uint8)


@pytest.mark.parametrize("fa,fb", PAIRS)
def test_acc_exact_rational_tiny_shapes_all_layouts(fa, fb):
    """Exact rational sums rounded to fp32 on tiny shapes, in all four storage
    layouts. Operand exponents are limited so that every partial sum is exact
    in fp64 (then the fp64 result rounds once to fp32 like the exact sum)."""
    rng = np.random.default_rng(100 + 4 * fa + fb)
    for trial in range(60):
        M, N, K = (int(v) for v in rng.integers(1, 6, size=3))
        lo_a, hi_a = (-9, 8) if fa == orc.E4M3 else (-8, 10)
        lo_b, hi_b = (-9, 8) if fb == orc.E4M3 else (-8, 10)
        A = _finite_codes(fa, rng, M * K, lo_a, hi_a).reshape(M, K)
        B = _finite_codes(fb, rng, K * N, lo_b, hi_b).reshape(K, N)
        dA = orc.decode(fa, A)
        dB = orc.decode(fb, B)
        ref = np.empty((M, N), np.float32)
        for i, j in itertools.product(range(M), range(N)):
            s = sum((Fraction(dA[i, k]) * Fraction(dB[k, j]) for k in range(K)), Fraction(0))
            ref[i, j] = np.float32(float(s))   # s fits in 53 bits: float(s) is exact
        for ta, tb in itertools.product((False, True), repeat=2):
            Ast = A.T.copy() if ta else A
            Bst = B.T.copy() if tb else B
            acc = orc.matmul_acc(Ast, fa, ta, Bst, fb, tb)
            assert np.array_equal(acc, ref), (trial, ta, tb)


def _int_grid_codes(fmt, rng, shape, vmax=8):
    """FP8 codes whose decoded values are small integers in [-vmax, vmax]."""
    table = {}
    for c in range(256):
        v = orc.decode(fmt, np.array([c]))[0]
        if math.isfinite(v) and v == int(v) and abs(v) <= vmax and c not in (0x80,):
            table.setdefault(int(v), c)
    keys = np.array(sorted(table))
    vals = rng.choice(keys, size=shape)
    codes = np.vectorize(table.get)(vals).astype(np.uint8)
    return codes, vals.astype(np.int64)


@pytest.mark.parametrize("fa,fb", [(orc.E4M3, orc.E4M3), (orc.E5M2, orc.E4M3)])
def test_acc_integer_grid_exact_at_large_k(fa, fb):
    """Integer-valued inputs: the sum is an integer below 2^24, so the exact
    result is known from int64 arithmetic."""
    rng = np.random.default_rng(5)
    A, Ai = _int_grid_codes(fa, rng, (32, 4096))
    B, Bi = _int_grid_codes(fb, rng, (4096, 24))
    acc = orc.matmul_acc(A, fa, False, B, fb, False)
    assert np.array_equal(acc, (Ai @ Bi).astype(np.float32))


def test_acc_at_matches_full_and_term_norm():
    rng = np.random.default_rng(9)
    A = torch.from_numpy(rng.standard_normal((40, 300)).astype(np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    B = torch.from_numpy(rng.standard_normal((300, 30)).astype(np.float32)).to(torch.float8_e5m2).view(torch.uint8).numpy()
    full = orc.matmul_acc(A, orc.E4M3, False, B, orc.E5M2, False)
    ii = rng.integers(0, 40, 200)
    jj = rng.integers(0, 30, 200)
    acc, tn = orc.matmul_acc_at(A, orc.E4M3, False, B, orc.E5M2, False, ii, jj)
    _, t1 = orc.matmul_acc_at(A, orc.E4M3, False, B, orc.E5M2, False, ii, jj, l1=True)
    assert np.array_equal(acc, full[ii, jj])
    dA, dB = torch_decode8(orc.E4M3, A), torch_decode8(orc.E5M2, B)
    terms = dA[ii, :] * dB[:, jj].T
    assert np.allclose(tn, np.sqrt((terms ** 2).sum(axis=1)), rtol=1e-12)
    assert np.allclose(t1, np.abs(terms).sum(axis=1), rtol=1e-12)


# ----------------------------------------------------------------------------- rescale / invariants

def test_rescale_exponent_closed_form_via_epilogue():
    # acc = 2^e_c * v, so amax of data is max|v|; out scale exponent is
    # e_a + e_b + e_c + floor(log2 amax)
    K = 4096  # e_c = 6
    for amax_v, e_r in [(1.0, 0), (1.999, 0), (2.0, 1), (3.5, 1), (0.5, -1), (0.26, -2), (448.0, 8)]:
        acc = np.array([amax_v * 64.0, -0.125, 0.0], np.float32)
        codes, e_out, amax = orc.matmul_epilogue(acc, 2.0 ** -3, 2.0 ** 5, K)
        assert amax == np.float32(amax_v)
        assert e_out == -3 + 5 + 6 + e_r
    # nothing to measure: zero, Inf, all NaN -> e_r = 0 (scale = propagated scale)
    for acc in ([0.0, -0.0], [np.inf, 1.0], [np.nan, np.nan]):
        _, e_out, _ = orc.matmul_epilogue(np.array(acc, np.float32), 1.0, 1.0, K)
        assert e_out == 6
    # NaN is ignored by amax
    _, e_out, amax = orc.matmul_epilogue(np.array([np.nan, 64.0 * 4], np.float32), 1.0, 1.0, K)
    assert amax == 4.0 and e_out == 6 + 2


def test_rescaled_amax_lands_in_target_binade():
    rng = np.random.default_rng(12)
    for t in (0, 3, 8):
        acc = (rng.standard_normal(5000) * 37.0).astype(np.float32)
        codes, e_out, amax = orc.matmul_epilogue(acc, 1.0, 1.0, 1, target_log2=t)
        m = np.abs(orc.decode(orc.E4M3, codes)).max()
        assert 2.0 ** t <= m <= 2.0 ** (t + 1)


def test_scale_clamped_to_e8m0_range():
    acc = np.array([1.0, 2.0], np.float32)
    _, e_out, _ = orc.matmul_epilogue(acc, 2.0 ** 100, 2.0 ** 100, 1, mode=orc.RESCALE_NONE)
    assert e_out == 127
    # the clamp moves the difference into the data, which then saturates
    codes, e_out, _ = orc.matmul_epilogue(acc, 2.0 ** 100, 2.0 ** 100, 1, mode=orc.RESCALE_NONE,
                                          out_fmt=orc.F16)
    assert e_out == 127 and list(codes) == [0x7BFF, 0x7BFF]


def _ulp_half(fmt, v):
    """Half the spacing of format fmt around |v| (a bound on RNE error)."""
    mant = {orc.E4M3: 3, orc.E5M2: 2}[fmt]
    emin = {orc.E4M3: -6, orc.E5M2: -14}[fmt]
    e = np.maximum(np.floor(np.log2(np.maximum(np.abs(v), 1e-300))), emin)
    return 0.5 * np.exp2(e - mant)


@pytest.mark.parametrize("fa,fb,out_fmt", [(orc.E4M3, orc.E4M3, orc.E4M3),
                                           (orc.E5M2, orc.E4M3, orc.E5M2),
                                           (orc.E4M3, orc.E5M2, orc.E5M2)])
def test_model_invariance_decoded_output_equals_unscaled_matmul(fa, fb, out_fmt):
    """dec(out) * s_out equals s_a*s_b*(A@B) up to the final rounding alone
    (Section 1: the transform does not change the graph's semantics)."""
    rng = np.random.default_rng(21)
    M, N, K = 48, 40, 300
    A = torch.from_numpy(rng.standard_normal((M, K)).astype(np.float32)).to(TORCH_F8[fa]).view(torch.uint8).numpy()
    B = torch.from_numpy(rng.standard_normal((K, N)).astype(np.float32)).to(TORCH_F8[fb]).view(torch.uint8).numpy()
    s_a, s_b = 2.0 ** -3, 2.0 ** 5
    codes, e_out, amax, acc = orc.matmul(A, fa, False, s_a, B, fb, False, s_b, out_fmt=out_fmt)
    exact = torch_decode8(fa, A) @ torch_decode8(fb, B) * s_a * s_b      # fp64, values exact
    got = orc.decode(out_fmt, codes) * 2.0 ** e_out
    data_exact = exact / 2.0 ** e_out
    err = np.abs(got - exact) / 2.0 ** e_out
    bound = _ulp_half(out_fmt, data_exact) + np.abs(data_exact) * 2.0 ** -23
    assert np.all(err <= bound)


@pytest.mark.parametrize("fmt", [orc.E4M3, orc.E5M2])
def test_pow2_rebalance_is_lossless_when_nothing_leaves_normal_range(fmt):
    """set_scaling by 2^k keeps decoded values bit-identical when no value
    leaves the normal range (Section 2: a power-of-two rescale is an
    exponent add)."""
    rng = np.random.default_rng(31)
    emax = 15 if fmt == orc.E4M3 else 30
    codes = rng.integers(0, 256, 4000).astype(np.uint8)
    exp_field = (codes >> (3 if fmt == orc.E4M3 else 2)) & (15 if fmt == orc.E4M3 else 31)
    for k in (-3, -1, 1, 2, 4):
        keep = (exp_field >= 1 + max(k, 0)) & (exp_field <= emax - 1 + min(k, 0))
        c = codes[keep]
        s_in = 2.0 ** 7
        out = orc.set_scaling(c, fmt, s_in, 7 + k, out_fmt=fmt)
        before = orc.decode(fmt, c) * s_in
        after = orc.decode(fmt, out) * 2.0 ** (7 + k)
        assert np.array_equal(before, after)


def test_rescale_of_already_unit_max_data_is_identity():
    rng = np.random.default_rng(41)
    x = rng.uniform(-1.8, 1.8, 1000).astype(np.float32)
    x[0] = 1.5
    codes = orc.cast(orc.E4M3, x)
    out, e_out, amax = orc.rescale(codes, orc.E4M3, 2.0 ** -4)
    assert e_out == -4 and np.array_equal(out, codes)


def test_rescale_f32_input_values_preserved_to_rounding():
    rng = np.random.default_rng(42)
    x = (rng.standard_normal(3000) * 1e-3).astype(np.float32)
    codes, e_out, amax = orc.rescale(x, orc.F32, 2.0 ** 3, out_fmt=orc.E4M3)
    assert amax == np.abs(x).max()
    got = orc.decode(orc.E4M3, codes) * 2.0 ** e_out
    data_exact = x.astype(np.float64) * 2.0 ** 3 / 2.0 ** e_out
    assert np.all(np.abs(got / 2.0 ** e_out - data_exact) <= _ulp_half(orc.E4M3, data_exact))


def test_cast_data_keeps_values_when_representable():
    codes = np.arange(256, dtype=np.uint8)
    out = orc.cast_data(codes, orc.E4M3, orc.F16)
    assert same_or_both_nan(orc.decode(orc.F16, out), orc.decode(orc.E4M3, codes))


# ----------------------------------------------------------------------------- hand-derived examples

def test_hand_derived_examples():
    with open(os.path.join(GOLDEN, "hand_examples.json")) as f:
        cases = json.load(f)["cases"]
    fmt_of = {"e4m3": orc.E4M3, "e5m2": orc.E5M2, "f16": orc.F16}
    for case in cases:
        A = np.array(case["a_codes"], dtype=np.uint8)
        B = np.array(case["b_codes"], dtype=np.uint8)
        codes, e_out, amax, acc = orc.matmul(
            A, fmt_of[case["a_fmt"]], False, 2.0 ** case["a_scale_log2"],
            B, fmt_of[case["b_fmt"]], False, 2.0 ** case["b_scale_log2"],
            mode=orc.RESCALE_AMAX if case["mode"] == "amax" else orc.RESCALE_NONE,
            target_log2=case.get("target_log2", 0), out_fmt=fmt_of[case["out_fmt"]])
        assert acc.tolist() == case["acc"], case["name"]
        assert codes.tolist() == case["out_codes"], case["name"]
        assert e_out == case["out_scale_log2"], case["name"]


def _pair(v):
    """[mantissa, exponent] of the epilogue goldens -> exact fp32."""
    return math.ldexp(float(v[0]), int(v[1]))


def test_epilogue_hand_examples_subnormal_accumulators():
    """Hand-derived epilogues of fp32-subnormal accumulators
    (tests/golden/epilogue_examples.json): the propagated data acc * 2^-e_c
    (Section 3.2) is an exact division, not an fp32 value of its own, so the
    statistic and every code come from acc through one power-of-two shift
    (Section 3.3 rebalance); rounding the data first changes scale and codes."""
    with open(os.path.join(GOLDEN, "epilogue_examples.json")) as f:
        cases = json.load(f)["cases"]
    fmt_of = {"e4m3": orc.E4M3, "e5m2": orc.E5M2, "f16": orc.F16}
    for c in cases:
        acc = np.array([[_pair(v) for v in row] for row in c["acc"]], dtype=np.float32)
        # the accumulators are what the derivation says: fp32 subnormals, exact
        assert np.all(np.abs(acc) < np.float32(2.0 ** -126)) and np.all(acc != 0), c["name"]
        codes, e_out, amax = orc.matmul_epilogue(
            acc, 2.0 ** c["a_scale_log2"], 2.0 ** c["b_scale_log2"], c["K"],
            orc.RESCALE_AMAX if c["mode"] == "amax" else orc.RESCALE_NONE, 0, True,
            fmt_of[c["out_fmt"]])
        assert codes.tolist() == c["out_codes"], (c["name"], codes.tolist())
        assert e_out == c["out_scale_log2"], (c["name"], e_out)
        assert amax == _pair(c["amax"]), (c["name"], amax)


def test_epilogue_is_one_rounding_of_the_exact_product_value():
    """Model invariance (Section 1: scaling leaves the computation unchanged)
    down to the fp32 subnormal range: each decoded output code times the
    output scale is the nearest E4M3 value (in output-scale units) of the
    exact value acc * s_a * s_b, whatever e_c the depth K gives."""
    rng = np.random.default_rng(23)
    units = rng.integers(-2 ** 20, 2 ** 20, 400)
    acc = np.ldexp(units.astype(np.float64), -149 - rng.integers(0, 4, 400)).astype(np.float32)
    for K in (1, 4, 64, 4096):
        codes, e_out, _ = orc.matmul_epilogue(acc, 2.0 ** 70, 2.0 ** 50, K)
        exact = acc.astype(np.float64) * 2.0 ** 120
        want = orc.cast(orc.E4M3, np.ldexp(exact, -e_out).astype(np.float32))
        # the shifted exact values are fp32 numbers (a power-of-two shift of
        # an fp32 value that stays normal), so casting them is one rounding
        assert np.array_equal(np.ldexp(np.ldexp(exact, -e_out).astype(np.float32).astype(np.float64),
                                       e_out), exact)
        assert np.array_equal(codes, want), K


def test_nan_sign_is_kept_through_decode_and_cast():
    """Reading R7: a NaN keeps its sign bit (as torch's float8 casts do)."""
    codes = np.array([0x7F, 0xFF], np.uint8)
    assert list(orc.cast_data(codes, orc.E4M3, orc.E4M3)) == [0x7F, 0xFF]
    assert list(orc.cast_data(codes, orc.E4M3, orc.F16)) == [0x7E00, 0xFE00]
    ref = torch.from_numpy(np.array([np.nan, -np.nan], np.float32)).to(torch.float8_e4m3fn)
    assert list(ref.view(torch.uint8).numpy()) == [0x7F, 0xFF]


# ------------------------------------------------------------------ delayed rescale

def test_delayed_hand_examples():
    """Delayed rescaling (Section 3.3): hand-derived cases, tests/golden/delayed_examples.json."""
    with open(os.path.join(GOLDEN, "delayed_examples.json")) as f:
        cases = json.load(f)["cases"]
    fmt_of = {"e4m3": orc.E4M3, "e5m2": orc.E5M2, "f16": orc.F16}
    for c in cases:
        acc = np.array(c["acc"], dtype=np.float32)
        codes, e_out, amax = orc.matmul_epilogue_delayed(
            acc, 2.0 ** c["a_scale_log2"], 2.0 ** c["b_scale_log2"], c["K"], c["amax_in"],
            saturate=c["saturate"], out_fmt=fmt_of[c["out_fmt"]])
        assert codes.tolist() == c["out_codes"], c["name"]
        assert e_out == c["out_scale_log2"], c["name"]
        assert amax == c["amax"], c["name"]


@pytest.mark.parametrize("out_fmt", [orc.E4M3, orc.E5M2, orc.F16])
@pytest.mark.parametrize("target", [0, 3])
def test_delayed_with_the_current_statistic_is_the_dynamic_rescale(out_fmt, target):
    """Fed this call's own amax, the delayed rescale is the dynamic one."""
    rng = np.random.default_rng(7 + out_fmt + 10 * target)
    acc = (rng.standard_normal((37, 29)) * 2.0 ** rng.integers(-6, 9, (37, 29))).astype(np.float32)
    K = 300
    dyn = orc.matmul_epilogue(acc, 2.0 ** -3, 2.0 ** 2, K, orc.RESCALE_AMAX, target, True, out_fmt)
    dl = orc.matmul_epilogue_delayed(acc, 2.0 ** -3, 2.0 ** 2, K, dyn[2], target, True, out_fmt)
    assert np.array_equal(dyn[0], dl[0]) and dyn[1] == dl[1] and dyn[2] == dl[2]


@pytest.mark.parametrize("stat", [0.0, float("inf"), float("nan")])
def test_delayed_without_a_statistic_is_the_static_rule(stat):
    """amax_in of 0, +Inf or NaN measures nothing: no rebalance (NONE mode)."""
    rng = np.random.default_rng(11)
    acc = (rng.standard_normal(500) * 40).astype(np.float32)
    ref = orc.matmul_epilogue(acc, 1.0, 0.5, 64, orc.RESCALE_NONE, 0, True, orc.E4M3)
    dl = orc.matmul_epilogue_delayed(acc, 1.0, 0.5, 64, stat, 0, True, orc.E4M3)
    assert np.array_equal(ref[0], dl[0]) and ref[1] == dl[1] and ref[2] == dl[2]


def test_delayed_stale_statistic_saturates_exactly_past_the_rounding_boundary():
    """A statistic 2^j too small scales the data up by 2^j, so the largest
    magnitudes leave the E4M3 range. The max code 0x7E (448) must then be
    exactly the elements with |data'| >= 432: from 432 (the tie between 416
    and 448, which goes to the even code 448) up to 464 they round to 448,
    above 464 they overflow and saturate to 448."""
    v = np.arange(1, 2001, dtype=np.float32) / 8.0          # 0.125 .. 250, exact
    acc = np.concatenate([v, -v])
    stat = 0.25                                              # far below the amax of 250
    codes, e_out, _ = orc.matmul_epilogue_delayed(acc, 1.0, 1.0, 1, stat, 0, True, orc.E4M3)
    e_r = -2
    scaled = np.abs(acc.astype(np.float64)) * 2.0 ** (-e_r)   # exact: 0.5 .. 1000
    sat = (codes & 0x7F) == 0x7E
    assert e_out == e_r
    assert 0 < sat.sum() < sat.size
    assert np.array_equal(sat, scaled >= 432.0)              # 432 is the midpoint of 416 and 448
