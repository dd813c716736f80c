"""CPU oracle for the Scalify scaled matmul path (arXiv 2407.17353) - Python side.

TEST INFRASTRUCTURE ONLY: imported by tests/, by __graft_entry__.smoke() and by
the cpu_baseline leg of bench.py, never by the product package. It wraps the
plain C oracle in ``scalify_oracle.c`` (table decode, exact nearest-search cast,
fp64 ascending-k accumulation) with numpy-facing helpers.

Every function states the passage of the paper it follows:
  * ScaledArray X = X_d * X_s, power-of-two scale held in fp32 (Section 2).
  * matmul scale rule: divide by a power of two rounded down from sqrt(K)
    (Section 3.2, Algorithm 3; independent-Gaussian assumption).
  * dynamic rescale: statistic (amax) -> power of two (rounded down) ->
    rebalance_scale (Section 3.3, Algorithm 4).
  * set_scaling / get_data_and_scale (Section 3.1); casts act on data only
    (Appendix A).
  * scaled add (Algorithm 3: sqrt of the sum of squared scales, rounded down)
    and activations f(x) = x * g(x) with the scale unchanged (Appendix C.1).
  * LayerNorm on the data component with output scale 1 (Appendix C.2) and
    its input gradient with a dynamic rescale (Section 4).

Parity pins for every function live in tests/test_oracle_pins.py.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

E4M3, E5M2, F16, F32 = 0, 1, 2, 3
RESCALE_NONE, RESCALE_AMAX, RESCALE_DELAYED = 0, 1, 2
ACT_NONE, ACT_RELU, ACT_GELU_TANH, ACT_SILU = 0, 1, 2, 3

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "scalify_oracle.c")
# SCALIFY_ORACLE_LIB names another build of the same source (e.g. one with
# the address and undefined-behaviour sanitizers) to load instead.
_LIB = os.environ.get("SCALIFY_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")

_lib = None


def build() -> str:
    """Compile the C oracle with gcc (plain IEEE arithmetic: no fast-math, no
    FMA contraction). Returns the path of the shared library."""
    cmd = ["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
           "-shared", "-fPIC", "-Wall", "-o", _LIB + ".tmp", _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(_LIB + ".tmp", _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB):
        build()
    lib = ctypes.CDLL(_LIB)
    c_i64, c_i32, c_int, c_f32, c_f64 = (ctypes.c_int64, ctypes.c_int32, ctypes.c_int,
                                         ctypes.c_float, ctypes.c_double)
    vp = ctypes.c_void_p
    lib.or_decode.argtypes = [c_int, ctypes.c_uint32]
    lib.or_decode.restype = c_f64
    lib.or_cast.argtypes = [c_int, c_int, c_f32]
    lib.or_cast.restype = ctypes.c_uint32
    lib.or_cast_array.argtypes = [c_int, c_int, vp, c_i64, vp]
    lib.or_matmul_scale_log2.argtypes = [c_i64]
    lib.or_matmul_scale_log2.restype = c_i32
    lib.or_floor_log2.argtypes = [c_f64]
    lib.or_floor_log2.restype = c_i32
    lib.or_matmul_acc.argtypes = [vp, c_int, c_int, c_i64, vp, c_int, c_int, c_i64,
                                  c_i64, c_i64, c_i64, vp]
    lib.or_matmul_acc_at.argtypes = [vp, c_int, c_int, c_i64, vp, c_int, c_int, c_i64,
                                     c_i64, vp, vp, c_i64, vp, vp, vp]
    lib.or_matmul_acc_mx.argtypes = [vp, c_int, c_int, c_i64, vp, c_int, c_int, c_i64,
                                     c_i64, c_i64, c_i64, vp, vp, c_i64, vp]
    lib.or_matmul_acc_mx.restype = c_int
    lib.or_matmul_acc_mx_at.argtypes = [vp, c_int, c_int, c_i64, vp, c_int, c_int, c_i64,
                                        c_i64, vp, vp, c_i64, vp, vp, c_i64, vp, vp]
    lib.or_matmul_acc_mx_at.restype = c_int
    lib.or_matmul_epilogue.argtypes = [vp, c_i64, c_f32, c_f32, c_i64, c_int, c_i32, c_int,
                                       c_int, vp, ctypes.POINTER(c_i32), ctypes.POINTER(c_f32)]
    lib.or_matmul_epilogue.restype = c_int
    lib.or_matmul_epilogue_delayed.argtypes = [vp, c_i64, c_f32, c_f32, c_i64, c_f32, c_i32, c_int,
                                                c_int, vp, vp, vp]
    lib.or_matmul_epilogue_delayed.restype = c_int
    lib.or_rescale.argtypes = [c_int, vp, c_i64, c_f32, c_int, c_i32, c_int, c_int, vp,
                               ctypes.POINTER(c_i32), ctypes.POINTER(c_f32)]
    lib.or_rescale.restype = c_int
    lib.or_set_scaling.argtypes = [c_int, vp, c_i64, c_f32, c_i32, c_int, c_int, vp]
    lib.or_set_scaling.restype = c_int
    lib.or_cast_data.argtypes = [c_int, vp, c_i64, c_int, c_int, vp]
    lib.or_gate.argtypes = [c_int, c_f64]
    lib.or_gate.restype = c_f64
    lib.or_add_scale_log2.argtypes = [c_i32, c_i32]
    lib.or_add_scale_log2.restype = c_i32
    lib.or_fused_pre.argtypes = [vp, c_i64, c_i64, c_f32, c_f32, c_i64, vp, c_int, c_i64, c_f32,
                                 c_int, vp, vp, ctypes.POINTER(c_i32), ctypes.POINTER(c_i32)]
    lib.or_fused_pre.restype = c_int
    lib.or_fused_pre_ch.argtypes = [vp, c_i64, c_i64, c_f32, c_f32, vp, vp, c_i64, vp, c_int, c_i64,
                                    c_f32, c_int, vp, vp, ctypes.POINTER(c_i32),
                                    ctypes.POINTER(c_i32)]
    lib.or_fused_pre_ch.restype = c_int
    lib.or_finish_pre.argtypes = [vp, c_i64, c_i32, c_i32, c_int, c_i32, c_f32, c_int, c_int, vp,
                                  ctypes.POINTER(c_f32)]
    lib.or_finish_pre.restype = c_i32
    lib.or_layernorm_fwd_pre.argtypes = [c_int, vp, c_i64, c_i64, vp, vp, c_f64, vp, vp, vp]
    lib.or_layernorm_bwd_pre.argtypes = [c_int, vp, c_int, vp, c_i64, c_i64, vp, c_f64, vp, vp, vp]
    lib.or_init()
    _lib = lib
    return lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _code_dtype(fmt: int):
    return {E4M3: np.uint8, E5M2: np.uint8, F16: np.uint16, F32: np.float32}[fmt]


# --------------------------------------------------------------------------- formats

_tables = {}


def decode(fmt: int, codes) -> np.ndarray:
    """Closed-form decode of FP8 (OCP E4M3 / E5M2) or FP16 codes to float64
    (Section 1 / Appendix A formats)."""
    lib = _load()
    codes = np.asarray(codes)
    if fmt not in _tables:
        tab_size = 65536 if fmt == F16 else 256
        _tables[fmt] = np.array([lib.or_decode(fmt, c) for c in range(tab_size)], dtype=np.float64)
    return _tables[fmt][codes.astype(np.int64)]


def cast(fmt: int, x, saturate: bool = True) -> np.ndarray:
    """Round fp32 values to FP8/FP16 codes: exact nearest search over the
    representable values, ties to the even code, OCP saturation rules
    (stage 2 of the two-stage quantization, Section 2)."""
    lib = _load()
    x = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    out = np.empty(x.shape, dtype=_code_dtype(fmt))
    lib.or_cast_array(fmt, int(bool(saturate)), _ptr(x), x.size, _ptr(out))
    return out


def matmul_scale_log2(K: int) -> int:
    """e_c = log2 of sqrt(K) rounded down to a power of two (Section 3.2)."""
    return int(_load().or_matmul_scale_log2(int(K)))


def floor_log2(x: float) -> int:
    return int(_load().or_floor_log2(float(x)))


# --------------------------------------------------------------------------- matmul

def _operand(codes: np.ndarray, trans: bool):
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    return codes, codes.shape[1]


def matmul_acc(A: np.ndarray, fa: int, ta: bool, B: np.ndarray, fb: int, tb: bool) -> np.ndarray:
    """fp32 accumulator of the FP8 dot_general: fp64 sum over ascending k of the
    exact products, rounded once to fp32.

    A is stored [M,K] (ta False) or [K,M] (ta True); B is stored [K,N]
    (tb False) or [N,K] (tb True)."""
    lib = _load()
    A, lda = _operand(A, ta)
    B, ldb = _operand(B, tb)
    M, K = (A.shape[1], A.shape[0]) if ta else A.shape
    K2, N = (B.shape[1], B.shape[0]) if tb else B.shape
    assert K == K2, (K, K2)
    acc = np.empty((M, N), dtype=np.float32)
    lib.or_matmul_acc(_ptr(A), fa, int(ta), lda, _ptr(B), fb, int(tb), ldb, M, N, K, _ptr(acc))
    return acc


def matmul_acc_at(A, fa, ta, B, fb, tb, ii, jj, l1=False):
    """Accumulator at sampled output positions (ii[p], jj[p]) and a norm of
    the product terms at each position: the l2 norm, or with l1=True the sum
    of their magnitudes."""
    lib = _load()
    A, lda = _operand(A, ta)
    B, ldb = _operand(B, tb)
    K = A.shape[0] if ta else A.shape[1]
    ii = np.ascontiguousarray(ii, dtype=np.int64)
    jj = np.ascontiguousarray(jj, dtype=np.int64)
    acc = np.empty(ii.shape, dtype=np.float32)
    t2 = np.empty(ii.shape, dtype=np.float64)
    t1 = np.empty(ii.shape, dtype=np.float64)
    lib.or_matmul_acc_at(_ptr(A), fa, int(ta), lda, _ptr(B), fb, int(tb), ldb, K,
                         _ptr(ii), _ptr(jj), ii.size, _ptr(acc), _ptr(t2), _ptr(t1))
    return acc, (t1 if l1 else t2)


def mx_block_scale_ld(K: int) -> int:
    """Row length (bytes) of an MX block-scale array for depth K: one byte
    per 32 k, padded to whole 128-k steps (4 bytes each)."""
    return 4 * ((K + 127) // 128)


def _mx_scales(sa, sb, M, N, K):
    sa = np.ascontiguousarray(sa, dtype=np.uint8)
    sb = np.ascontiguousarray(sb, dtype=np.uint8)
    ld = sa.shape[1]
    assert sa.shape[0] == M and sb.shape == (N, ld) and ld >= (K + 31) // 32, (sa.shape, sb.shape)
    return sa, sb, ld


def matmul_acc_mx(A, fa, ta, B, fb, tb, sa, sb) -> np.ndarray:
    """fp32 accumulator of the FP8 dot_general with MX block scales
    (Section 2: block scaling formats as scales broadcastable to the data):
    sa[i, k // 32] and sb[j, k // 32] are E8M0 bytes (value 2^(byte - 127))
    multiplying A[i, k] and B[k, j]; fp64 sum over ascending k, one rounding
    to fp32. sa is [M][ld], sb [N][ld], ld >= ceil(K / 32). Raises on an
    0xFF (NaN) byte among those used."""
    lib = _load()
    A, lda = _operand(A, ta)
    B, ldb = _operand(B, tb)
    M, K = (A.shape[1], A.shape[0]) if ta else A.shape
    K2, N = (B.shape[1], B.shape[0]) if tb else B.shape
    assert K == K2, (K, K2)
    sa, sb, ld = _mx_scales(sa, sb, M, N, K)
    acc = np.empty((M, N), dtype=np.float32)
    if lib.or_matmul_acc_mx(_ptr(A), fa, int(ta), lda, _ptr(B), fb, int(tb), ldb, M, N, K,
                            _ptr(sa), _ptr(sb), ld, _ptr(acc)):
        raise ValueError("0xFF is not an E8M0 scale")
    return acc


def matmul_acc_mx_at(A, fa, ta, B, fb, tb, sa, sb, ii, jj):
    """matmul_acc_mx at sampled positions (ii[p], jj[p]), with the sum of
    the magnitudes of the scaled product terms at each."""
    lib = _load()
    A, lda = _operand(A, ta)
    B, ldb = _operand(B, tb)
    M, K = (A.shape[1], A.shape[0]) if ta else A.shape
    N = B.shape[0] if tb else B.shape[1]
    sa, sb, ld = _mx_scales(sa, sb, M, N, K)
    ii = np.ascontiguousarray(ii, dtype=np.int64)
    jj = np.ascontiguousarray(jj, dtype=np.int64)
    acc = np.empty(ii.shape, dtype=np.float32)
    t1 = np.empty(ii.shape, dtype=np.float64)
    if lib.or_matmul_acc_mx_at(_ptr(A), fa, int(ta), lda, _ptr(B), fb, int(tb), ldb, K,
                               _ptr(sa), _ptr(sb), ld, _ptr(ii), _ptr(jj), ii.size,
                               _ptr(acc), _ptr(t1)):
        raise ValueError("0xFF is not an E8M0 scale")
    return acc, t1


def matmul_epilogue(acc: np.ndarray, s_a: float, s_b: float, K: int, mode: int = RESCALE_AMAX,
                    target_log2: int = 0, saturate: bool = True, out_fmt: int = E4M3):
    """Scale propagation (Section 3.2) + dynamic amax rescale (Section 3.3) +
    cast (Section 2, stage 2) applied to an fp32 accumulator.

    Returns (codes, e_out, amax): output scale is 2**e_out; amax is
    max |acc * 2^-e_c| over non-NaN elements."""
    lib = _load()
    acc = np.ascontiguousarray(acc, dtype=np.float32)
    out = np.empty(acc.shape, dtype=_code_dtype(out_fmt))
    e_out = ctypes.c_int32(0)
    amax = ctypes.c_float(0)
    rc = lib.or_matmul_epilogue(_ptr(acc), acc.size, s_a, s_b, int(K), mode, target_log2,
                                int(bool(saturate)), out_fmt, _ptr(out),
                                ctypes.byref(e_out), ctypes.byref(amax))
    if rc != 0:
        raise ValueError("input scales must be finite powers of two")
    return out, int(e_out.value), float(amax.value)


def matmul_epilogue_delayed(acc: np.ndarray, s_a: float, s_b: float, K: int, amax_in: float,
                            target_log2: int = 0, saturate: bool = True, out_fmt: int = E4M3):
    """Delayed rescaling (Section 3.3): scale propagation and cast as in
    matmul_epilogue, with the rescale exponent taken from amax_in, the
    statistic recorded by an earlier call. Returns (codes, e_out, amax) where
    amax is this call's statistic (max |acc * 2^-e_c|), for the next call."""
    lib = _load()
    acc = np.ascontiguousarray(acc, dtype=np.float32)
    out = np.empty(acc.shape, dtype=_code_dtype(out_fmt))
    e_out = ctypes.c_int32(0)
    amax = ctypes.c_float(0)
    rc = lib.or_matmul_epilogue_delayed(_ptr(acc), acc.size, s_a, s_b, int(K), float(amax_in),
                                        target_log2, int(bool(saturate)), out_fmt, _ptr(out),
                                        ctypes.byref(e_out), ctypes.byref(amax))
    if rc != 0:
        raise ValueError("input scales must be finite powers of two")
    return out, int(e_out.value), float(amax.value)


def matmul(A, fa, ta, s_a, B, fb, tb, s_b, mode=RESCALE_AMAX, target_log2=0, saturate=True,
           out_fmt=E4M3):
    """Full scaled matmul on ScaledArray operands: accumulate, then epilogue.
    Returns (codes, e_out, amax, acc)."""
    acc = matmul_acc(A, fa, ta, B, fb, tb)
    K = A.shape[0] if ta else A.shape[1]
    codes, e_out, amax = matmul_epilogue(acc, s_a, s_b, K, mode, target_log2, saturate, out_fmt)
    return codes, e_out, amax, acc


# --------------------------------------------------------------------------- fused add / activation

def gate(act: int, x: float) -> float:
    """Gating function g of f(x) = x * g(x) (Appendix C.1), fp64."""
    return float(_load().or_gate(int(act), float(x)))


def add_scale_log2(e1: int, e2: int) -> int:
    """Scale exponent of a scaled add (Algorithm 3): sqrt(s1^2 + s2^2)
    rounded down to a power of two."""
    return int(_load().or_add_scale_log2(int(e1), int(e2)))


def fused_pre(acc: np.ndarray, s_a: float, s_b: float, K: int, residual=None,
              act: int = ACT_NONE, ch_a=None, ch_b=None):
    """Pre-cast value of the matmul epilogue with a fused scaled add and
    activation (Algorithm 3 add rule, Appendix C.1 activation rule).

    residual: None or (codes, fmt, scale): codes [M,N] or [1,N] (one row
    repeated, a bias) of format fmt with scalar scale `scale`.
    ch_a / ch_b: None or channel scales (powers of two), one per row of A
    ([M]) / per column of B ([N]) (Section 2: a scale broadcastable to the
    data), folded into w by one power-of-two product of acc.
    Returns (w, y64, e_w, e_cc): w fp32 [M,N] with true value w * 2^e_w,
    y64 the fp64 value before w's last rounding, and e_cc such that the
    rescale statistic is taken over w * 2^-e_cc."""
    lib = _load()
    acc = np.ascontiguousarray(acc, dtype=np.float32)
    M, N = acc.shape
    w = np.empty((M, N), dtype=np.float32)
    y64 = np.empty((M, N), dtype=np.float64)
    e_w = ctypes.c_int32(0)
    e_cc = ctypes.c_int32(0)
    ca = None if ch_a is None else np.ascontiguousarray(ch_a, dtype=np.float32).reshape(-1)
    cb = None if ch_b is None else np.ascontiguousarray(ch_b, dtype=np.float32).reshape(-1)
    assert ca is None or ca.size == M
    assert cb is None or cb.size == N
    if residual is None:
        codes_p, fmt, ld, scale = None, 0, 0, 1.0
    else:
        codes, fmt, scale = residual
        codes = np.ascontiguousarray(codes, dtype=_code_dtype(fmt))
        assert codes.shape in ((M, N), (1, N)), codes.shape
        ld = 0 if codes.shape[0] == 1 and M != 1 else N
        codes_p = _ptr(codes)
    rc = lib.or_fused_pre_ch(_ptr(acc), M, N, s_a, s_b, _ptr(ca) if ca is not None else None,
                             _ptr(cb) if cb is not None else None, int(K), codes_p, int(fmt), ld,
                             float(scale), int(act), _ptr(w), _ptr(y64), ctypes.byref(e_w),
                             ctypes.byref(e_cc))
    if rc != 0:
        raise ValueError("scales must be finite powers of two")
    return w, y64, int(e_w.value), int(e_cc.value)


def finish_pre(w: np.ndarray, e_w: int, e_cc: int, mode: int = RESCALE_AMAX, target_log2: int = 0,
               amax_in: float = 0.0, saturate: bool = True, out_fmt: int = E4M3):
    """Rescale (Section 3.3: amax, or the delayed statistic amax_in) and cast
    (Section 2, stage 2) of pre-cast values w whose true value is w * 2^e_w.
    Returns (codes, e_out, amax) with amax = max |w * 2^-e_cc| (non-NaN)."""
    lib = _load()
    w = np.ascontiguousarray(w, dtype=np.float32)
    out = np.empty(w.shape, dtype=_code_dtype(out_fmt))
    amax = ctypes.c_float(0)
    e_out = lib.or_finish_pre(_ptr(w), w.size, int(e_w), int(e_cc), int(mode), int(target_log2),
                              float(amax_in), int(bool(saturate)), int(out_fmt), _ptr(out),
                              ctypes.byref(amax))
    return out, int(e_out), float(amax.value)


def matmul_epilogue_fused(acc, s_a, s_b, K, residual=None, act=ACT_NONE, mode=RESCALE_AMAX,
                          target_log2=0, amax_in=0.0, saturate=True, out_fmt=E4M3,
                          ch_a=None, ch_b=None):
    """Matmul epilogue with the channel scales, the fused scaled add and the
    activation, then the rescale and cast. Returns (codes, e_out, amax, w, y64)."""
    w, y64, e_w, e_cc = fused_pre(acc, s_a, s_b, K, residual, act, ch_a, ch_b)
    codes, e_out, amax = finish_pre(w, e_w, e_cc, mode, target_log2, amax_in, saturate, out_fmt)
    return codes, e_out, amax, w, y64


# --------------------------------------------------------------------------- LayerNorm

def _f32_or_none(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float32)


def layernorm_fwd_pre(x, in_fmt: int, gamma=None, beta=None, eps: float = 1e-5):
    """Scaled LayerNorm forward on the data component (Appendix C.2): per row,
    xhat = (x - mean) / (std + eps), y = xhat * gamma + beta, output scale 1.
    x: codes (or fp32 values for F32) [R, D]. Returns (y64, mean, std), fp64."""
    lib = _load()
    x = np.ascontiguousarray(x, dtype=_code_dtype(in_fmt))
    R, D = x.shape
    y = np.empty((R, D), dtype=np.float64)
    mu = np.empty(R, dtype=np.float64)
    sd = np.empty(R, dtype=np.float64)
    g, b = _f32_or_none(gamma), _f32_or_none(beta)
    lib.or_layernorm_fwd_pre(int(in_fmt), _ptr(x), R, D, _ptr(g) if g is not None else None,
                             _ptr(b) if b is not None else None, float(eps), _ptr(y), _ptr(mu),
                             _ptr(sd))
    return y, mu, sd


def layernorm_fwd(x, in_fmt: int, gamma=None, beta=None, eps: float = 1e-5, saturate: bool = True,
                  out_fmt: int = E4M3):
    """Forward with the output cast: y rounded to fp32, then to out_fmt with
    scale 1 (Appendix C.2). Returns (codes, y64, mean, std)."""
    y64, mu, sd = layernorm_fwd_pre(x, in_fmt, gamma, beta, eps)
    codes, e_out, _ = finish_pre(y64.astype(np.float32), 0, 0, RESCALE_NONE, 0, 0.0, saturate,
                                 out_fmt)
    assert e_out == 0
    return codes, y64, mu, sd


def layernorm_bwd_pre(dy, dy_fmt: int, x, x_fmt: int, gamma=None, eps: float = 1e-5):
    """Gradient of the data-component LayerNorm (Appendix C.2) for an
    upstream gradient with data dy: returns (dx64, dgamma, dbeta) in fp64;
    the true input gradient is dx64 * s_dy / X_s, the parameter gradients
    are in units of s_dy."""
    lib = _load()
    dy = np.ascontiguousarray(dy, dtype=_code_dtype(dy_fmt))
    x = np.ascontiguousarray(x, dtype=_code_dtype(x_fmt))
    assert dy.shape == x.shape
    R, D = x.shape
    dx = np.empty((R, D), dtype=np.float64)
    dg = np.empty(D, dtype=np.float64)
    db = np.empty(D, dtype=np.float64)
    g = _f32_or_none(gamma)
    lib.or_layernorm_bwd_pre(int(dy_fmt), _ptr(dy), int(x_fmt), _ptr(x), R, D,
                             _ptr(g) if g is not None else None, float(eps), _ptr(dx), _ptr(dg),
                             _ptr(db))
    return dx, dg, db


def layernorm_bwd(dy, dy_fmt, s_dy, x, x_fmt, s_x, gamma=None, eps=1e-5, mode=RESCALE_AMAX,
                  target_log2=0, saturate=True, out_fmt=E5M2):
    """LayerNorm input gradient with its dynamic rescale (Section 4, the
    LayerNorm backward rescale; Section 3.3): the ScaledArray (dx, s_dy / s_x)
    rebalanced by the amax rule and cast. Returns (codes, e_out, amax, dx64,
    dgamma, dbeta)."""
    dx64, dg, db = layernorm_bwd_pre(dy, dy_fmt, x, x_fmt, gamma, eps)
    e_in = int(_load().or_floor_log2(float(s_dy))) - int(_load().or_floor_log2(float(s_x)))
    codes, e_out, amax = finish_pre(dx64.astype(np.float32), e_in, 0, mode, target_log2, 0.0,
                                    saturate, out_fmt)
    return codes, e_out, amax, dx64, dg, db


# --------------------------------------------------------------------------- rescale / cast

def rescale(data: np.ndarray, in_fmt: int, s_in: float, mode: int = RESCALE_AMAX,
            target_log2: int = 0, saturate: bool = True, out_fmt: int = E4M3):
    """Dynamic rescale of a ScaledArray (Section 3.3): amax of the decoded data
    -> power of two rounded down -> rebalance_scale -> cast. Returns
    (codes, e_out, amax)."""
    lib = _load()
    data = np.ascontiguousarray(data, dtype=_code_dtype(in_fmt))
    out = np.empty(data.shape, dtype=_code_dtype(out_fmt))
    e_out = ctypes.c_int32(0)
    amax = ctypes.c_float(0)
    rc = lib.or_rescale(in_fmt, _ptr(data), data.size, s_in, mode, target_log2,
                        int(bool(saturate)), out_fmt, _ptr(out), ctypes.byref(e_out),
                        ctypes.byref(amax))
    if rc != 0:
        raise ValueError("input scale must be a finite power of two")
    return out, int(e_out.value), float(amax.value)


def set_scaling(data: np.ndarray, in_fmt: int, s_in: float, e_new: int, saturate: bool = True,
                out_fmt: int = E4M3) -> np.ndarray:
    """set_scaling (Section 3.1): output scale 2^e_new, data rescaled by the
    ratio of old and new scales, then cast."""
    lib = _load()
    data = np.ascontiguousarray(data, dtype=_code_dtype(in_fmt))
    out = np.empty(data.shape, dtype=_code_dtype(out_fmt))
    rc = lib.or_set_scaling(in_fmt, _ptr(data), data.size, s_in, e_new, int(bool(saturate)),
                            out_fmt, _ptr(out))
    if rc != 0:
        raise ValueError("bad scale")
    return out


def cast_data(data: np.ndarray, in_fmt: int, out_fmt: int, saturate: bool = True) -> np.ndarray:
    """Cast operator on the data component only; the scale is unchanged
    (Appendix A)."""
    lib = _load()
    data = np.ascontiguousarray(data, dtype=_code_dtype(in_fmt))
    out = np.empty(data.shape, dtype=_code_dtype(out_fmt))
    lib.or_cast_data(in_fmt, _ptr(data), data.size, int(bool(saturate)), out_fmt, _ptr(out))
    return out
