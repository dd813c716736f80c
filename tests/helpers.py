"""Shared helpers of the GPU parity tests: run the HIP path through the C ABI
and compare it with the CPU oracle under the parity contract:

  P1  codes, output scale and amax equal the oracle epilogue applied to the
      GPU's own fp32 accumulator (exact);
  P2  the GPU accumulator equals the oracle's fp64-then-fp32 sum within
      1e-5 * sqrt(K) * max(|acc|, ||a_i||_2 ||b_j||_2) per element: the
      relative error of a dot product measured against its Cauchy-Schwarz
      bound, the scale its rounding error is classically bounded by (the
      FP8 MFMA adds each group of products in a window 14 bits wide below
      the group's largest product, so errors scale with the largest terms,
      not with |acc|);
  P3  end-to-end codes equal the oracle's except where a value inside the P2
      band around the oracle accumulator rounds to the GPU's code (the two
      sums straddle a rounding boundary); for FP8 outputs such a flip moves
      the code by one position in value order; flips are counted, recorded
      and bounded per case.
"""
from __future__ import annotations

import json
import math
import os
import sys

import numpy as np
import torch

from oracle import oracle as orc
from paper_2407_17353_amd import binding as sc

FMT = {0: "e4m3", 1: "e5m2", 2: "f16"}


def say(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def pad16(x: int) -> int:
    return max(16, (x + 15) // 16 * 16)


def stored_with_padding(codes: torch.Tensor, device, pad_byte: int = 0x7F) -> torch.Tensor:
    """Copy a stored code matrix [R, C] to the device inside [R, pad16(C)]
    storage whose padding bytes hold pad_byte (NaN in both FP8 formats), so a
    kernel that reads past the logical columns would be caught."""
    R, C = codes.shape
    st = torch.full((R, pad16(C)), pad_byte, dtype=torch.uint8, device=device)
    st[:, :C] = codes.to(device)
    return st[:, :C]


def gpu_matmul(A_st, fa, ta, sa_log2, B_st, fb, tb, sb_log2, fout, mode=sc.RESCALE_AMAX,
               target=0, saturate=True, device="cuda", want_acc=True, pad_byte=0x7F):
    """Run scalify_matmul on stored code matrices (CPU or device uint8
    tensors). Returns (codes[M,N] numpy, e_out, amax, acc numpy or None)."""
    a = sc.ScaledArray(stored_with_padding(A_st, device, pad_byte), fa,
                       sc.scale_tensor(sa_log2, device) if sa_log2 is not None else None, ta)
    b = sc.ScaledArray(stored_with_padding(B_st, device, pad_byte), fb,
                       sc.scale_tensor(sb_log2, device) if sb_log2 is not None else None, tb)
    M, K = a.shape
    _, N = b.shape
    out = sc.empty_scaled(M, N, fout, device)
    acc = torch.empty((M, N), dtype=torch.float32, device=device) if want_acc else None
    amax = torch.empty(1, dtype=torch.float32, device=device)
    sc.scalify_matmul(a, b, out, rescale=mode, target_log2=target, saturate=saturate,
                      acc_out=acc, amax_out=amax)
    torch.cuda.synchronize()
    codes = out.data.cpu().numpy()
    if fout == sc.F16:
        codes = codes.view(np.uint16)
    s = float(out.scale.item())
    e_out = int(math.frexp(s)[1] - 1)
    assert s == 2.0 ** e_out
    return codes.copy(), e_out, float(amax.item()), (acc.cpu().numpy() if want_acc else None)


def check_p1(codes, e_out, amax, acc, K, sa_log2, sb_log2, fout, mode=sc.RESCALE_AMAX, target=0,
             saturate=True):
    """P1: the oracle epilogue on the GPU accumulator gives identical codes,
    scale and amax."""
    ref_codes, ref_e, ref_amax = orc.matmul_epilogue(
        acc, 2.0 ** (sa_log2 or 0), 2.0 ** (sb_log2 or 0), K, mode, target, saturate, fout)
    assert e_out == ref_e, (e_out, ref_e)
    assert np.array_equal(np.float32(amax), np.float32(ref_amax)) or (np.isnan(amax) and np.isnan(ref_amax)), (amax, ref_amax)
    bad = np.flatnonzero(codes.ravel() != ref_codes.ravel())
    assert bad.size == 0, f"P1: {bad.size} code mismatches, first {bad[:5]} " \
        f"gpu {codes.ravel()[bad[:5]]} ref {ref_codes.ravel()[bad[:5]]} acc {acc.ravel()[bad[:5]]}"
    return ref_e


def acc_tolerance(ref, term_norm, K):
    return 1e-5 * math.sqrt(K) * np.maximum(np.abs(ref.astype(np.float64)), term_norm)


def operand_norms(A, fa, ta, B, fb, tb):
    """l2 norms of the logical rows of A and columns of B (decoded values,
    non-finite entries left out)."""
    dA = orc.decode(fa, A)
    dB = orc.decode(fb, B)
    dA = np.where(np.isfinite(dA), dA, 0.0)
    dB = np.where(np.isfinite(dB), dB, 0.0)
    ra = np.sqrt((dA ** 2).sum(axis=0 if ta else 1))
    cb = np.sqrt((dB ** 2).sum(axis=1 if tb else 0))
    return ra, cb


def check_p2_full(acc_gpu, A_st, fa, ta, B_st, fb, tb):
    """P2 on every element (oracle accumulates the whole matrix)."""
    A = A_st.cpu().numpy()
    B = B_st.cpu().numpy()
    ref = orc.matmul_acc(A, fa, ta, B, fb, tb)
    K = A.shape[0] if ta else A.shape[1]
    ra, cb = operand_norms(A, fa, ta, B, fb, tb)
    scale = np.outer(ra, cb)
    return _compare_acc(acc_gpu, ref, scale, K), ref, scale


def check_p2_sampled(acc_gpu, A_st, fa, ta, B_st, fb, tb, n_samples=65536, seed=0):
    """P2 on a seeded sample of output positions, each summed exactly by the
    oracle (for sizes where the full oracle is too slow)."""
    A = A_st.cpu().numpy()
    B = B_st.cpu().numpy()
    M, N = acc_gpu.shape
    K = A.shape[0] if ta else A.shape[1]
    rng = np.random.default_rng(seed)
    ii = rng.integers(0, M, n_samples)
    jj = rng.integers(0, N, n_samples)
    # always include the corners and edges of the matrix
    ii = np.concatenate([ii, [0, 0, M - 1, M - 1]])
    jj = np.concatenate([jj, [0, N - 1, 0, N - 1]])
    ref, _ = orc.matmul_acc_at(A, fa, ta, B, fb, tb, ii, jj)
    ra, cb = operand_norms(A, fa, ta, B, fb, tb)
    scale = ra[ii] * cb[jj]
    return _compare_acc(acc_gpu[ii, jj], ref, scale, K), ii, jj, ref, scale


def _compare_acc(gpu, ref, tn, K):
    gpu = np.asarray(gpu, dtype=np.float32)
    nan_g, nan_r = np.isnan(gpu), np.isnan(ref)
    assert np.array_equal(nan_g, nan_r), "NaN pattern differs"
    fin = ~nan_r & np.isfinite(ref)
    assert np.array_equal(gpu[~fin & ~nan_r], ref[~fin & ~nan_r]), "Inf pattern differs"
    err = np.abs(gpu[fin].astype(np.float64) - ref[fin].astype(np.float64))
    tol = acc_tolerance(ref[fin], tn[fin] if np.ndim(tn) else tn, K)
    worst = float((err / np.maximum(tol, 1e-300)).max()) if err.size else 0.0
    assert np.all(err <= tol), f"P2: worst err/tol {worst}"
    return worst


def code_ordinal(fmt, codes):
    """Position of FP8 codes in the order of their values (sign-magnitude
    codes: +-0 share position 0, the next representable magnitude is 1)."""
    c = np.asarray(codes).astype(np.int64)
    mag = c & 0x7F
    return np.where(c & 0x80, -mag, mag)


def record(kind: str, **fields):
    """Append one JSON line to the file named by SCALIFY_PARITY_LOG, if set
    (the measured flip counts behind the P3 bounds)."""
    path = os.environ.get("SCALIFY_PARITY_LOG")
    if path:
        with open(path, "a") as f:
            f.write(json.dumps({"kind": kind, **fields}) + "\n")


def check_p3(codes_gpu, acc_ref, term_norm, K, shift, fout, saturate=True, max_flips=0,
             max_multi=0, name=""):
    """P3: end-to-end codes against the oracle's own accumulator. A code may
    differ from the oracle's only if it is the rounding of a value inside the
    P2 tolerance band around the oracle accumulator (the two sums fall on
    different sides of a rounding boundary). For FP8 outputs a flip moves the
    code by one position in value order wherever the band holds at most one
    rounding boundary; flips of more than one position ("multi-code") are
    possible only where cancellation makes the band wider than the code
    spacing at the sum, and are counted apart. Both counts are recorded and
    bounded (max_flips, max_multi): their rates are a property of the MFMA's
    accumulation, largest for FP16 outputs and for heavy-range gradients."""
    acc_ref = np.asarray(acc_ref, dtype=np.float32).ravel()
    g = np.asarray(codes_gpu).ravel()
    ref_codes = orc.cast(fout, np.ldexp(acc_ref, -shift).astype(np.float32), saturate)
    bad = np.flatnonzero(g != ref_codes)
    multi = 0
    if bad.size:
        tol = acc_tolerance(acc_ref[bad], np.asarray(term_norm).ravel()[bad], K)
        lo = orc.cast(fout, np.ldexp(acc_ref[bad] - tol, -shift).astype(np.float32), saturate)
        hi = orc.cast(fout, np.ldexp(acc_ref[bad] + tol, -shift).astype(np.float32), saturate)
        vg, vlo, vhi = orc.decode(fout, g[bad]), orc.decode(fout, lo), orc.decode(fout, hi)
        ok = (vlo <= vg) & (vg <= vhi)
        assert np.all(ok), f"P3: code outside the tolerance band at {bad[~ok][:5]}"
        if fout != sc.F16:
            step = np.abs(code_ordinal(fout, g[bad]) - code_ordinal(fout, ref_codes[bad]))
            span = code_ordinal(fout, hi) - code_ordinal(fout, lo)  # boundaries inside the band
            narrow = span <= 1
            assert np.all(step[narrow] <= 1), \
                f"P3: flips of more than one code inside narrow bands at {bad[narrow & (step > 1)][:5]}"
            multi = int(np.count_nonzero(step > 1))
    record("p3", name=name, K=int(K), fout=FMT[fout], n=int(g.size), flips=int(bad.size),
           multi=multi)
    say(f"  P3 {name}: {bad.size} flips of {g.size} ({FMT[fout]}), {multi} multi-code")
    assert bad.size <= max_flips, f"P3: {bad.size} flips of {g.size}, bound {max_flips}"
    assert multi <= max_multi, f"P3: {multi} multi-code flips, bound {max_multi}"
    return int(bad.size)
