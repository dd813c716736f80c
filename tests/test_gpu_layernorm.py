"""GPU parity of the scaled LayerNorm (Appendix C.2) and of its input gradient
with the dynamic rescale (Section 4), through the C ABI, against the oracle.

The kernels export the value they cast (`pre_out`: y in the forward, dx
before the rescale in the backward). Checks:
  L1  that value against the oracle's fp64 one, within the fp32 rounding of
      the row statistics (forward: 1.5e-6 (|gamma| (1 + |xhat|) + |beta|),
      about 25 fp32 ulps; backward: 1e-6 times the sum of the magnitudes of
      the terms of dx);
  L2  codes, output scale (and the backward's amax) exactly equal to the
      oracle's cast / rescale of the kernel's own value;
  L3  dgamma and dbeta against the oracle within 2e-5 of the sums of the
      magnitudes of their terms.
"""
import contextlib
import math
import os

import numpy as np
import pytest
import torch

from oracle import oracle as orc
from paper_2407_17353_amd import binding as sc
from tests.helpers import say

pytestmark = pytest.mark.gpu

DEV = "cuda"
FMT_NAMES = {sc.E4M3: "e4m3", sc.E5M2: "e5m2", sc.F16: "f16", sc.F32: "f32"}


def _values(R, D, seed, loc=0.0, scale=1.0, spread=None):
    g = torch.Generator().manual_seed(seed)
    x = torch.randn((R, D), generator=g, dtype=torch.float32) * scale + loc
    if spread is not None:
        x = x * torch.exp2(torch.randint(-spread, spread + 1, (R, 1), generator=g).float())
    return x.numpy()


def _codes(vals, fmt):
    """Storage of `vals` in format fmt (numpy): codes, or fp32 for F32."""
    if fmt == sc.F32:
        return np.ascontiguousarray(vals, dtype=np.float32)
    return orc.cast(fmt, vals)


def _device(codes, fmt, ld=None):
    """Padded device rows (ld a multiple of 16 bytes) holding `codes`."""
    R, D = codes.shape
    per16 = {sc.E4M3: 16, sc.E5M2: 16, sc.F16: 8, sc.F32: 4}[fmt]
    ld = ld or max(per16, (D + per16 - 1) // per16 * per16)
    tdt = {sc.E4M3: torch.uint8, sc.E5M2: torch.uint8, sc.F16: torch.int16, sc.F32: torch.float32}[fmt]
    st = torch.zeros((R, ld), dtype=tdt, device=DEV)
    src = torch.from_numpy(codes.view(np.int16) if fmt == sc.F16 else codes)
    st[:, :D] = src.to(DEV)
    return st[:, :D]


def _to_np(t, fmt):
    a = t.cpu().numpy()
    return a.view(np.uint16) if fmt == sc.F16 else a


def run_fwd(xc, xfmt, out_fmt, gamma=None, beta=None, eps=1e-5, sat=True):
    R, D = xc.shape
    x = sc.ScaledArray(_device(xc, xfmt), xfmt, sc.scale_tensor(7, DEV))
    out = sc.ScaledArray(_device(np.zeros((R, D), dtype=np.float32 if out_fmt == sc.F32 else
                                          (np.uint16 if out_fmt == sc.F16 else np.uint8)), out_fmt),
                         out_fmt, torch.full((1,), 3.0, device=DEV))
    pre = torch.empty((R, D), dtype=torch.float32, device=DEV)
    g = torch.from_numpy(gamma).to(DEV) if gamma is not None else None
    b = torch.from_numpy(beta).to(DEV) if beta is not None else None
    sc.scalify_layernorm_fwd(x, out, gamma=g, beta=b, eps=eps, saturate=sat, pre_out=pre)
    torch.cuda.synchronize()
    return _to_np(out.data, out_fmt), float(out.scale.item()), pre.cpu().numpy()


def check_fwd(run, xc, xfmt, out_fmt, gamma, beta, eps, sat=True):
    codes, scale, pre = run
    assert scale == 1.0
    y64, mu, sd = orc.layernorm_fwd_pre(xc, xfmt, gamma, beta, eps)
    xh, _, _ = orc.layernorm_fwd_pre(xc, xfmt, None, None, eps)
    gm = np.abs(gamma.astype(np.float64)) if gamma is not None else 1.0
    bm = np.abs(beta.astype(np.float64)) if beta is not None else 0.0
    tol = 1.5e-6 * (gm * (1.0 + np.abs(xh)) + bm)
    nan = np.isnan(y64)
    assert np.array_equal(np.isnan(pre), nan), "L1: NaN pattern"
    err = np.abs(pre[~nan].astype(np.float64) - y64[~nan])
    assert np.all(err <= tol[~nan] if np.ndim(tol) else err <= tol), \
        f"L1: worst err/tol {float((err / np.broadcast_to(tol, y64.shape)[~nan]).max())}"
    ref, e_out, _ = orc.finish_pre(pre, 0, 0, orc.RESCALE_NONE, 0, 0.0, sat, out_fmt)
    assert e_out == 0
    bad = np.flatnonzero(codes.ravel() != ref.ravel())
    assert bad.size == 0, f"L2: {bad.size} code mismatches, first {bad[:5]}"
    return float((err / np.broadcast_to(tol, y64.shape)[~nan]).max()) if err.size else 0.0


FWD_CASES = [
    # (R, D, x fmt, out fmt, affine, eps)
    (1, 1, sc.F16, sc.E4M3, False, 1e-5),
    (3, 17, sc.F32, sc.E5M2, True, 1e-5),
    (64, 768, sc.F16, sc.E4M3, True, 1e-5),
    (33, 1000, sc.E4M3, sc.F16, True, 0.0),
    (5, 8192, sc.F16, sc.E4M3, True, 1e-5),
    (7, 4097, sc.E5M2, sc.E5M2, False, 0.5),
    (300, 4096, sc.F16, sc.E4M3, True, 1e-5),
    (1030, 256, sc.F32, sc.F16, True, 1e-3),
    # rows of 2049 .. 4096 FP16 / FP8 elements: the pipelined kernel (several
    # rows per wave, a ragged last chunk)
    (5000, 2112, sc.F16, sc.E5M2, True, 1e-5),
    (11, 3001, sc.E4M3, sc.F16, True, 0.0),
    (2100, 2049, sc.E5M2, sc.E4M3, False, 1e-5),
]


@pytest.mark.parametrize("case", FWD_CASES, ids=lambda c: f"{c[0]}x{c[1]}-{FMT_NAMES[c[2]]}-"
                                                          f"{FMT_NAMES[c[3]]}-{'aff' if c[4] else 'noaff'}")
def test_layernorm_fwd_parity(case):
    R, D, xfmt, ofmt, affine, eps = case
    say(f"case ln fwd {case}")
    rng = np.random.default_rng(R * 7 + D)
    xc = _codes(_values(R, D, 100 + D, loc=0.7, scale=3.0, spread=6), xfmt)
    gamma = (rng.standard_normal(D) * 0.5 + 1.0).astype(np.float32) if affine else None
    beta = (rng.standard_normal(D) * 0.2).astype(np.float32) if affine else None
    run = run_fwd(xc, xfmt, ofmt, gamma, beta, eps)
    worst = check_fwd(run, xc, xfmt, ofmt, gamma, beta, eps)
    say(f"  ok, worst err/tol {worst:.3g}")


def test_layernorm_fwd_specials_and_in_place():
    """Constant rows (std 0: y = beta), a NaN row, saturation off, and out
    written over x (same rows, same element size)."""
    say("case ln fwd specials")
    R, D = 6, 300
    vals = _values(R, D, 5)
    vals[1] = 2.5
    vals[2, 17] = np.nan
    xc = _codes(vals, sc.F16)
    beta = np.linspace(-3, 3, D).astype(np.float32)
    gamma = np.full(D, 300.0, dtype=np.float32)
    run = run_fwd(xc, sc.F16, sc.E4M3, gamma, beta, 1e-5, sat=False)
    check_fwd(run, xc, sc.F16, sc.E4M3, gamma, beta, 1e-5, sat=False)
    assert np.isnan(run[2][2]).all()
    # in place: F16 -> F16 over the same storage
    xd = _device(xc, sc.F16)
    x = sc.ScaledArray(xd, sc.F16, sc.scale_tensor(0, DEV))
    out = sc.ScaledArray(xd, sc.F16, torch.empty(1, device=DEV))
    sc.scalify_layernorm_fwd(x, out, eps=1e-5)
    sep = run_fwd(xc, sc.F16, sc.F16, None, None, 1e-5)
    torch.cuda.synchronize()
    assert np.array_equal(_to_np(xd, sc.F16), sep[0])


def run_bwd(dyc, dyfmt, sdy, xc, xfmt, sx, out_fmt, gamma=None, eps=1e-5, mode=sc.RESCALE_AMAX,
            target=0, sat=True):
    R, D = xc.shape
    dy = sc.ScaledArray(_device(dyc, dyfmt), dyfmt, sc.scale_tensor(sdy, DEV))
    x = sc.ScaledArray(_device(xc, xfmt), xfmt, sc.scale_tensor(sx, DEV))
    dx = sc.ScaledArray(_device(np.zeros((R, D), dtype=np.uint16 if out_fmt == sc.F16 else np.uint8),
                                out_fmt), out_fmt, torch.empty(1, device=DEV))
    pre = torch.empty((R, D), dtype=torch.float32, device=DEV)
    dg = torch.empty(D, dtype=torch.float32, device=DEV)
    db = torch.empty(D, dtype=torch.float32, device=DEV)
    amax = torch.empty(1, dtype=torch.float32, device=DEV)
    g = torch.from_numpy(gamma).to(DEV) if gamma is not None else None
    sc.scalify_layernorm_bwd(dy, x, dx, gamma=g, eps=eps, rescale=mode, target_log2=target,
                             saturate=sat, dgamma=dg, dbeta=db, amax_out=amax, pre_out=pre)
    torch.cuda.synchronize()
    s = float(dx.scale.item())
    e_out = int(math.frexp(s)[1] - 1)
    assert s == 2.0 ** e_out
    return (_to_np(dx.data, out_fmt), e_out, float(amax.item()), pre.cpu().numpy(),
            dg.cpu().numpy(), db.cpu().numpy())


def check_bwd(run, dyc, dyfmt, sdy, xc, xfmt, sx, out_fmt, gamma, eps, mode, target=0, sat=True):
    codes, e_out, amax, pre, dg, db = run
    dx64, dg64, db64 = orc.layernorm_bwd_pre(dyc, dyfmt, xc, xfmt, gamma, eps)
    # magnitudes of the terms of dx, for its rounding bound
    xh, mu, sd = orc.layernorm_fwd_pre(xc, xfmt, None, None, eps)
    dyv = dyc.astype(np.float64) if dyfmt == sc.F32 else orc.decode(dyfmt, dyc)
    xv = xc.astype(np.float64) if xfmt == sc.F32 else orc.decode(xfmt, xc)
    gam = gamma.astype(np.float64) if gamma is not None else 1.0
    g = dyv * gam
    s = (sd + eps)[:, None]
    mg = np.abs(g).mean(axis=1, keepdims=True)
    mgx = np.abs(g * xh).mean(axis=1, keepdims=True)
    c_sig = np.where(sd[:, None] > 0, np.abs(xv - mu[:, None]) / np.where(sd[:, None] > 0, sd[:, None], 1.0), 0.0)
    tol = 1e-6 * (np.abs(g) + mg + c_sig * mgx + np.abs(dx64)) / s
    nan = np.isnan(dx64)
    assert np.array_equal(np.isnan(pre), nan), "L1: NaN pattern"
    err = np.abs(pre[~nan].astype(np.float64) - dx64[~nan])
    worst = float((err / np.maximum(tol[~nan], 1e-300)).max()) if err.size else 0.0
    assert np.all(err <= tol[~nan]), f"L1: worst err/tol {worst}"
    e_in = int(math.frexp(2.0 ** sdy)[1] - 1) - int(math.frexp(2.0 ** sx)[1] - 1)
    ref, ref_e, ref_amax = orc.finish_pre(pre, e_in, 0, mode, target, 0.0, sat, out_fmt)
    assert e_out == ref_e, (e_out, ref_e)
    assert np.float32(amax) == np.float32(ref_amax), (amax, ref_amax)
    bad = np.flatnonzero(codes.ravel() != ref.ravel())
    assert bad.size == 0, f"L2: {bad.size} code mismatches, first {bad[:5]}"
    # L3
    fin = np.isfinite(dg64)
    tg = 2e-5 * np.abs(dyv * xh).sum(axis=0)
    tb = 2e-5 * np.abs(dyv).sum(axis=0)
    assert np.all(np.abs(dg[fin] - dg64[fin]) <= tg[fin] + 1e-30), "L3: dgamma"
    assert np.all(np.abs(db[fin] - db64[fin]) <= tb[fin] + 1e-30), "L3: dbeta"
    return worst


BWD_CASES = [
    # (R, D, dy fmt, x fmt, out fmt, affine, eps, mode)
    (1, 1, sc.F16, sc.F16, sc.E5M2, False, 1e-5, sc.RESCALE_AMAX),
    (3, 17, sc.F32, sc.F32, sc.E4M3, True, 1e-5, sc.RESCALE_AMAX),
    (64, 768, sc.E5M2, sc.F16, sc.E5M2, True, 1e-5, sc.RESCALE_AMAX),
    (33, 1000, sc.F16, sc.E4M3, sc.F16, True, 0.0, sc.RESCALE_NONE),
    (5, 8192, sc.E5M2, sc.F16, sc.E5M2, True, 1e-5, sc.RESCALE_AMAX),
    (7, 4097, sc.E4M3, sc.E5M2, sc.E4M3, False, 0.5, sc.RESCALE_AMAX),
    (1030, 256, sc.F16, sc.F32, sc.F16, True, 1e-3, sc.RESCALE_AMAX),
    # rows of 2049 .. 4096 FP16 / FP8 elements: the pipelined statistics
    # kernel (several rows per wave, ragged last chunks, D = 4096 whole)
    (3000, 4096, sc.E5M2, sc.F16, sc.E5M2, True, 1e-5, sc.RESCALE_AMAX),
    (2500, 2112, sc.F16, sc.E4M3, sc.E4M3, True, 1e-5, sc.RESCALE_AMAX),
    (9, 3001, sc.E4M3, sc.E5M2, sc.F16, False, 0.0, sc.RESCALE_NONE),
    (17, 2049, sc.F16, sc.F16, sc.E5M2, True, 1e-5, sc.RESCALE_AMAX),
]


@pytest.mark.parametrize("case", BWD_CASES, ids=lambda c: f"{c[0]}x{c[1]}-{FMT_NAMES[c[2]]}-"
                                                          f"{FMT_NAMES[c[3]]}-{FMT_NAMES[c[4]]}-m{c[7]}")
def test_layernorm_bwd_parity(case):
    R, D, dyfmt, xfmt, ofmt, affine, eps, mode = case
    say(f"case ln bwd {case}")
    rng = np.random.default_rng(R * 11 + D)
    xc = _codes(_values(R, D, 200 + D, loc=-0.3, scale=2.0, spread=5), xfmt)
    dyc = _codes(_values(R, D, 300 + D, spread=8), dyfmt)
    gamma = (rng.standard_normal(D) * 0.5 + 1.0).astype(np.float32) if affine else None
    for sdy, sx in [(0, 0), (-9, 4)]:
        run = run_bwd(dyc, dyfmt, sdy, xc, xfmt, sx, ofmt, gamma, eps, mode)
        worst = check_bwd(run, dyc, dyfmt, sdy, xc, xfmt, sx, ofmt, gamma, eps, mode)
        say(f"  scales {sdy},{sx} ok, worst err/tol {worst:.3g}")


def test_layernorm_bwd_specials_targets_in_place():
    """Constant rows (std 0), a NaN in dy (the statistic skips it), targets,
    saturation off, and dx written over dy."""
    say("case ln bwd specials")
    R, D = 9, 520
    xv = _values(R, D, 11)
    xv[3] = -1.25
    dyv = _values(R, D, 12, spread=3)
    dyv[5, 7] = np.nan
    xc, dyc = _codes(xv, sc.F16), _codes(dyv, sc.F16)
    for target, sat in [(0, True), (3, False), (-2, True)]:
        run = run_bwd(dyc, sc.F16, 2, xc, sc.F16, -1, sc.E5M2, None, 0.25, sc.RESCALE_AMAX,
                      target, sat)
        check_bwd(run, dyc, sc.F16, 2, xc, sc.F16, -1, sc.E5M2, None, 0.25, sc.RESCALE_AMAX,
                  target, sat)
    # in place over dy (F16 -> F16)
    dyd = _device(dyc, sc.F16)
    dy = sc.ScaledArray(dyd, sc.F16, sc.scale_tensor(0, DEV))
    x = sc.ScaledArray(_device(xc, sc.F16), sc.F16, sc.scale_tensor(0, DEV))
    dx = sc.ScaledArray(dyd, sc.F16, torch.empty(1, device=DEV))
    sc.scalify_layernorm_bwd(dy, x, dx, eps=0.25)
    sep = run_bwd(dyc, sc.F16, 0, xc, sc.F16, 0, sc.F16, None, 0.25)
    torch.cuda.synchronize()
    assert np.array_equal(_to_np(dyd, sc.F16), sep[0])


def test_layernorm_empty():
    say("case ln empty")
    for R, D in [(0, 16), (0, 0)]:
        x = sc.ScaledArray(torch.zeros((R, max(D, 16)), dtype=torch.int16, device=DEV)[:, :D],
                           sc.F16, None)
        out = sc.ScaledArray(torch.zeros((R, max(D, 16)), dtype=torch.uint8, device=DEV)[:, :D],
                             sc.E4M3, torch.zeros(1, device=DEV))
        sc.scalify_layernorm_fwd(x, out)
        torch.cuda.synchronize()
        assert out.scale.item() == 1.0


def test_layernorm_transformer_layer_full_size():
    """The LayerNorm of the LLaMA-7B-size layer at 16384 tokens (d = 4096):
    FP16 residual stream -> E4M3 forward; E5M2 gradient -> E5M2 input
    gradient with the dynamic rescale. L1/L2 on every element, L3 on every
    parameter."""
    R, D = 16384, 4096
    say("case ln full 16384x4096")
    rng = np.random.default_rng(9)
    xc = _codes(_values(R, D, 901, loc=0.1, scale=1.5), sc.F16)
    gamma = (rng.standard_normal(D) * 0.2 + 1.0).astype(np.float32)
    beta = (rng.standard_normal(D) * 0.1).astype(np.float32)
    run = run_fwd(xc, sc.F16, sc.E4M3, gamma, beta, 1e-5)
    w = check_fwd(run, xc, sc.F16, sc.E4M3, gamma, beta, 1e-5)
    say(f"  fwd ok, worst err/tol {w:.3g}")
    dyc = _codes(_values(R, D, 902, scale=2.0 ** -6, spread=4), sc.E5M2)
    run = run_bwd(dyc, sc.E5M2, 0, xc, sc.F16, 0, sc.E5M2, gamma, 1e-5)
    w = check_bwd(run, dyc, sc.E5M2, 0, xc, sc.F16, 0, sc.E5M2, gamma, 1e-5, sc.RESCALE_AMAX)
    say(f"  bwd ok, worst err/tol {w:.3g}")


@contextlib.contextmanager
def _env(**kw):
    old = {k: os.environ.get(k) for k in kw}
    os.environ.update({k: str(v) for k, v in kw.items()})
    try:
        yield
    finally:
        for k, v in old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


@pytest.mark.parametrize("R,D,xfmt,dyfmt,ofmt", [(640, 4096, sc.F16, sc.E5M2, sc.E4M3),
                                                 (257, 3001, sc.E4M3, sc.F16, sc.E5M2),
                                                 (96, 2049, sc.E5M2, sc.E4M3, sc.F16)],
                         ids=lambda v: str(v))
def test_single_read_kernels_equal_the_multi_pass_ones(R, D, xfmt, dyfmt, ofmt):
    """The forward and the backward statistics that read each row once
    (rows of 2049..4096 FP16 / FP8 elements) give the same bits as the
    multi-pass kernels (SCALIFY_LN_SINGLE_READ=0): same arithmetic, same
    order."""
    say(f"case layernorm single-read vs multi-pass R={R} D={D}")
    rng = np.random.default_rng(R + D)
    xc = _codes(_values(R, D, 300 + D, loc=0.3, scale=2.0, spread=5), xfmt)
    dyc = _codes(_values(R, D, 400 + D, scale=0.5, spread=4), dyfmt)
    gamma = (rng.standard_normal(D) * 0.5 + 1.0).astype(np.float32)
    beta = (rng.standard_normal(D) * 0.2).astype(np.float32)
    f1 = run_fwd(xc, xfmt, ofmt, gamma, beta, 1e-5)
    b1 = run_bwd(dyc, dyfmt, -2, xc, xfmt, 3, ofmt, gamma, 1e-5)
    with _env(SCALIFY_LN_SINGLE_READ=0):
        f0 = run_fwd(xc, xfmt, ofmt, gamma, beta, 1e-5)
        b0 = run_bwd(dyc, dyfmt, -2, xc, xfmt, 3, ofmt, gamma, 1e-5)
    assert np.array_equal(f1[0], f0[0]) and f1[1] == f0[1]
    assert np.array_equal(f1[2].view(np.uint32), f0[2].view(np.uint32))
    assert np.array_equal(b1[0], b0[0]) and b1[1] == b0[1] and b1[2] == b0[2]
    for k in (3, 4, 5):
        assert np.array_equal(b1[k].view(np.uint32), b0[k].view(np.uint32))
    check_fwd(f1, xc, xfmt, ofmt, gamma, beta, 1e-5)
