"""Pins of the oracle's scaled LayerNorm (Appendix C.2: normalize the data
component, output scale 1) and of its input gradient with the dynamic
rescale (Section 4).

Routes that do not go through the oracle's own formulas: hand-derived rows,
the invariances of a mean-variance normalization (shift, and scale up to
eps), moments of the output, central finite differences of the forward for
every gradient, and the properties the gradient of a shift- and
scale-invariant map must have.
"""
import math

import numpy as np
import pytest

from oracle import oracle as orc


def _rows(rng, R, D, loc=0.0, scale=1.0):
    return (rng.standard_normal((R, D)) * scale + loc).astype(np.float32)


def test_hand_derived_row():
    """x = [1, 2, 3, 4]: mean 5/2, variance (9/4 + 1/4 + 1/4 + 9/4)/4 = 5/4,
    so xhat = (x - 5/2) / (sqrt(5/4) + eps); gamma = 2, beta = 1/2 apply."""
    x = np.array([[1, 2, 3, 4]], dtype=np.float32)
    eps = 1.0 / 1024
    y, mu, sd = orc.layernorm_fwd_pre(x, orc.F32, np.full(4, 2.0), np.full(4, 0.5), eps)
    assert mu[0] == 2.5 and abs(sd[0] - math.sqrt(1.25)) < 1e-15
    want = np.array([-1.5, -0.5, 0.5, 1.5]) / (math.sqrt(1.25) + eps) * 2.0 + 0.5
    assert np.allclose(y[0], want, rtol=1e-15, atol=1e-15)


def test_output_moments_and_invariances():
    """mean(xhat) = 0 and mean(xhat^2) = sigma^2 / (sigma + eps)^2 per row;
    adding a constant to a row changes nothing; scaling a row by a power of
    two changes nothing when eps = 0 (the scale invariance the paper uses to
    normalize X_d instead of X)."""
    rng = np.random.default_rng(1)
    x = _rows(rng, 9, 257, loc=3.0, scale=2.0)
    for eps in (0.0, 1e-3):
        y, mu, sd = orc.layernorm_fwd_pre(x, orc.F32, eps=eps)
        assert np.allclose(y.mean(axis=1), 0.0, atol=1e-13)
        assert np.allclose((y ** 2).mean(axis=1), sd ** 2 / (sd + eps) ** 2, rtol=1e-12)
    y0, _, _ = orc.layernorm_fwd_pre(x, orc.F32, eps=0.0)
    y1, _, _ = orc.layernorm_fwd_pre(x + np.float32(0.5), orc.F32, eps=0.0)
    y2, _, _ = orc.layernorm_fwd_pre(x * np.float32(8.0), orc.F32, eps=0.0)
    assert np.allclose(y0, y1, atol=1e-6)          # x + 0.5 rounds in fp32
    assert np.allclose(y0, y2, rtol=1e-14, atol=1e-14)


def test_constant_row_gives_beta():
    x = np.full((2, 16), 3.0, dtype=np.float32)
    beta = np.linspace(-1, 1, 16).astype(np.float32)
    y, mu, sd = orc.layernorm_fwd_pre(x, orc.F32, None, beta, 1e-5)
    assert np.all(sd == 0.0) and np.array_equal(y, np.tile(beta.astype(np.float64), (2, 1)))


@pytest.mark.parametrize("fmt", [orc.E4M3, orc.E5M2, orc.F16])
def test_input_codes_are_decoded(fmt):
    """Code inputs normalize their decoded values (checked against the F32 path)."""
    rng = np.random.default_rng(2 + fmt)
    codes = orc.cast(fmt, _rows(rng, 5, 64))
    vals = orc.decode(fmt, codes).astype(np.float32)
    a = orc.layernorm_fwd_pre(codes, fmt)[0]
    b = orc.layernorm_fwd_pre(vals, orc.F32)[0]
    assert np.array_equal(a, b)


def _loss(x, dy, gamma, beta, eps):
    y, _, _ = orc.layernorm_fwd_pre(x, orc.F32, gamma, beta, eps)
    return float((y * dy).sum())


@pytest.mark.parametrize("eps", [0.0, 0.05])
def test_gradients_match_central_differences(eps):
    """dL/dx, dL/dgamma, dL/dbeta of L = sum(y * dy) against central
    differences of the forward (step 2^-12, fp64 values exactly representable
    in fp32 inputs, error O(h^2)). A dropped term or a sign slip in the
    backward formula fails by orders of magnitude."""
    rng = np.random.default_rng(3)
    R, D = 3, 8
    x = _rows(rng, R, D)
    dy = _rows(rng, R, D)
    gamma = (rng.standard_normal(D) * 0.5 + 1.0).astype(np.float32)
    beta = rng.standard_normal(D).astype(np.float32)
    dx, dg, db = orc.layernorm_bwd_pre(dy, orc.F32, x, orc.F32, gamma, eps)
    h = 2.0 ** -12
    for r in range(R):
        for j in range(D):
            xp, xm = x.copy(), x.copy()
            xp[r, j] += np.float32(h)
            xm[r, j] -= np.float32(h)
            num = (_loss(xp, dy, gamma, beta, eps) - _loss(xm, dy, gamma, beta, eps)) / (2 * h)
            assert abs(num - dx[r, j]) < 2e-5 * (1 + abs(num)), (r, j, num, dx[r, j])
    for j in range(D):
        gp, gm = gamma.copy(), gamma.copy()
        gp[j] += np.float32(h)
        gm[j] -= np.float32(h)
        num = (_loss(x, dy, gp, beta, eps) - _loss(x, dy, gm, beta, eps)) / (2 * h)
        assert abs(num - dg[j]) < 2e-5 * (1 + abs(num))
        bp, bm = beta.copy(), beta.copy()
        bp[j] += np.float32(h)
        bm[j] -= np.float32(h)
        num = (_loss(x, dy, gamma, bp, eps) - _loss(x, dy, gamma, bm, eps)) / (2 * h)
        assert abs(num - db[j]) < 2e-5 * (1 + abs(num))


def test_gradient_is_orthogonal_to_the_invariances():
    """The forward ignores a constant added to a row, so every row of the
    input gradient sums to 0; with eps = 0 it also ignores a scaling of the
    row, so sum_j dx_j * (x_j - mean) = 0."""
    rng = np.random.default_rng(4)
    x = _rows(rng, 6, 300, loc=-2.0, scale=3.0)
    dy = _rows(rng, 6, 300)
    dx, _, _ = orc.layernorm_bwd_pre(dy, orc.F32, x, orc.F32, None, 1e-3)
    assert np.allclose(dx.sum(axis=1), 0.0, atol=1e-12)
    dx0, _, _ = orc.layernorm_bwd_pre(dy, orc.F32, x, orc.F32, None, 0.0)
    c = x.astype(np.float64) - x.astype(np.float64).mean(axis=1, keepdims=True)
    assert np.allclose((dx0 * c).sum(axis=1), 0.0, atol=1e-10)


def test_constant_row_gradient():
    """A constant row has sigma = 0: the gradient is (g - mean(g)) / eps."""
    x = np.full((1, 8), 2.0, dtype=np.float32)
    dy = np.arange(8, dtype=np.float32)[None, :]
    dx, _, _ = orc.layernorm_bwd_pre(dy, orc.F32, x, orc.F32, None, 0.25)
    assert np.allclose(dx[0], (np.arange(8) - 3.5) / 0.25, rtol=1e-15)


@pytest.mark.parametrize("out_fmt", [orc.E4M3, orc.E5M2, orc.F16])
def test_gradient_rescale_lands_in_the_target_binade(out_fmt):
    """The dynamic rescale of the input gradient: the ScaledArray
    (dx, s_dy / s_x) is rebalanced so that its amax lies in [1, 2), and the
    decoded output times its scale is the true gradient up to the cast."""
    rng = np.random.default_rng(5 + out_fmt)
    x = _rows(rng, 4, 128, scale=4.0)
    dy = (_rows(rng, 4, 128) * 2.0 ** -20).astype(np.float32)
    s_dy, s_x = 2.0 ** -3, 2.0 ** 5
    codes, e_out, amax, dx64, _, _ = orc.layernorm_bwd(dy, orc.F32, s_dy, x, orc.F32, s_x,
                                                       out_fmt=out_fmt)
    e_in = -3 - 5
    assert 2.0 ** (e_out - e_in) <= np.abs(dx64).max() * (1 + 1e-6) < 2.0 ** (e_out - e_in + 1)
    true = dx64 * s_dy / s_x
    got = orc.decode(out_fmt, codes) * 2.0 ** e_out
    rel = 2.0 ** -3 if out_fmt == orc.E4M3 else (2.0 ** -2 if out_fmt == orc.E5M2 else 2.0 ** -10)
    big = np.abs(true) > 2.0 ** (e_out - 6)
    assert np.all(np.abs(got[big] - true[big]) <= rel * np.abs(true[big]))
