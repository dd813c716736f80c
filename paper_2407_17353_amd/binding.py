"""Python binding of libscalify.so (include/scalify.h): argument marshalling only.

Every step of the scaled matmul, rescale and cast runs in the HIP kernels of
the library; this module turns torch device tensors into the C structs, picks
the current HIP stream, allocates workspaces with torch and raises on a
non-OK status. There is no fallback: if the library is missing, importing it
raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import torch

E4M3, E5M2, F16, F32 = 0, 1, 2, 3
RESCALE_NONE, RESCALE_AMAX, RESCALE_DELAYED = 0, 1, 2
ACT_NONE, ACT_RELU, ACT_GELU_TANH, ACT_SILU = 0, 1, 2, 3

STATUS_NAMES = {0: "SCALIFY_OK", 1: "SCALIFY_ERR_NULL", 2: "SCALIFY_ERR_DTYPE",
                3: "SCALIFY_ERR_SHAPE", 4: "SCALIFY_ERR_LAYOUT", 5: "SCALIFY_ERR_ALIGN",
                6: "SCALIFY_ERR_WORKSPACE", 7: "SCALIFY_ERR_VALUE", 8: "SCALIFY_ERR_HIP"}

# storage element type of each format (codes are carried as raw bits)
STORAGE_DTYPE = {E4M3: torch.uint8, E5M2: torch.uint8, F16: torch.int16, F32: torch.float32}

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libscalify.so")


class ScalifyError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {STATUS_NAMES.get(status, status)} "
                         f"({string_of(status)})")


class CScaledArray(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("scale", ctypes.c_void_p), ("dtype", ctypes.c_int32),
                ("trans", ctypes.c_int32), ("rows", ctypes.c_int64), ("cols", ctypes.c_int64),
                ("ld", ctypes.c_int64)]


class CMatmulOpts(ctypes.Structure):
    _fields_ = [("out_dtype", ctypes.c_int32), ("rescale", ctypes.c_int32),
                ("target_log2", ctypes.c_int32), ("saturate", ctypes.c_int32),
                ("acc_out", ctypes.c_void_p), ("amax_out", ctypes.c_void_p),
                ("events", ctypes.c_void_p), ("amax_in", ctypes.c_void_p),
                ("residual", ctypes.POINTER(CScaledArray)), ("activation", ctypes.c_int32),
                ("pre_out", ctypes.c_void_p), ("a_channel_scale", ctypes.c_void_p),
                ("b_channel_scale", ctypes.c_void_p), ("a_block_scale", ctypes.c_void_p),
                ("b_block_scale", ctypes.c_void_p)]


EXPORTED = ("scalify_matmul_scale_log2", "scalify_matmul_workspace_size",
            "scalify_matmul_workspace_size_opts", "scalify_matmul",
            "scalify_rescale_workspace_size", "scalify_rescale", "scalify_cast",
            "scalify_set_scaling", "scalify_status_string", "scalify_layernorm_fwd",
            "scalify_layernorm_bwd_workspace_size", "scalify_layernorm_bwd",
            "scalify_mx_packed_bytes", "scalify_mx_pack_block_scales",
            "scalify_matmul_noalloc")

_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libscalify.so (built by paper_2407_17353_amd/build.py). Raises
    FileNotFoundError when it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise FileNotFoundError(f"{path} is missing: run paper_2407_17353_amd/build.py")
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    lib.scalify_matmul_scale_log2.argtypes = [i64]
    lib.scalify_matmul_scale_log2.restype = i32
    lib.scalify_mx_packed_bytes.argtypes = [i64, i64]
    lib.scalify_mx_packed_bytes.restype = i64
    lib.scalify_mx_pack_block_scales.argtypes = [vp, i64, i64, i64, vp, vp]
    lib.scalify_mx_pack_block_scales.restype = ctypes.c_int
    lib.scalify_matmul_workspace_size.argtypes = [i64, i64, i32, i32]
    lib.scalify_matmul_workspace_size.restype = ctypes.c_size_t
    lib.scalify_matmul_workspace_size_opts.argtypes = [i64, i64, P(CMatmulOpts)]
    lib.scalify_matmul_workspace_size_opts.restype = ctypes.c_size_t
    lib.scalify_matmul.argtypes = [P(CScaledArray), P(CScaledArray), P(CScaledArray),
                                   P(CMatmulOpts), vp, ctypes.c_size_t, vp]
    lib.scalify_matmul.restype = ctypes.c_int
    lib.scalify_matmul_noalloc.argtypes = [P(CScaledArray), P(CScaledArray), P(CScaledArray),
                                           P(CMatmulOpts), vp]
    lib.scalify_matmul_noalloc.restype = ctypes.c_int
    lib.scalify_rescale_workspace_size.argtypes = [i64]
    lib.scalify_rescale_workspace_size.restype = ctypes.c_size_t
    lib.scalify_rescale.argtypes = [P(CScaledArray), P(CScaledArray), i32, i32, i32, vp,
                                    ctypes.c_size_t, vp]
    lib.scalify_rescale.restype = ctypes.c_int
    lib.scalify_cast.argtypes = [P(CScaledArray), P(CScaledArray), i32, vp]
    lib.scalify_cast.restype = ctypes.c_int
    lib.scalify_set_scaling.argtypes = [P(CScaledArray), P(CScaledArray), i32, i32, vp]
    lib.scalify_set_scaling.restype = ctypes.c_int
    f32 = ctypes.c_float
    lib.scalify_layernorm_fwd.argtypes = [P(CScaledArray), vp, vp, f32, P(CScaledArray), i32, vp, vp]
    lib.scalify_layernorm_fwd.restype = ctypes.c_int
    lib.scalify_layernorm_bwd_workspace_size.argtypes = [i64, i64]
    lib.scalify_layernorm_bwd_workspace_size.restype = ctypes.c_size_t
    lib.scalify_layernorm_bwd.argtypes = [P(CScaledArray), P(CScaledArray), vp, f32, P(CScaledArray),
                                          vp, vp, i32, i32, i32, vp, vp, vp, ctypes.c_size_t, vp]
    lib.scalify_layernorm_bwd.restype = ctypes.c_int
    lib.scalify_status_string.argtypes = [i32]
    lib.scalify_status_string.restype = ctypes.c_char_p
    _lib = lib
    return lib


def string_of(status: int) -> str:
    return load_library().scalify_status_string(int(status)).decode()


@dataclass
class ScaledArray:
    """A ScaledArray (data, scale) with value = decode(data) * scale
    (Section 2 of the paper). `data` is the STORED matrix as a 2-D tensor
    whose rows are contiguous (stride(1) == 1; stride(0) is the leading
    dimension); with trans=True it stores the transpose of the logical
    matrix. `scale` is a one-element float32 device tensor or None (scale 1)."""
    data: torch.Tensor
    fmt: int
    scale: Optional[torch.Tensor] = None
    trans: bool = False

    @property
    def shape(self):
        r, c = self.data.shape
        return (c, r) if self.trans else (r, c)

    def c_struct(self) -> CScaledArray:
        d = self.data
        if d.dim() != 2:
            raise ValueError("ScaledArray data must be 2-D")
        if d.shape[0] * d.shape[1] > 0 and d.stride(1) != 1:
            raise ValueError("ScaledArray rows must be contiguous")
        rows, cols = self.shape
        ld = d.stride(0) if d.numel() else 0
        return CScaledArray(d.data_ptr() if d.numel() else None,
                            self.scale.data_ptr() if self.scale is not None else None,
                            int(self.fmt), int(bool(self.trans)), rows, cols, ld)


def _stream_handle(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def _check(status: int, where: str):
    if status != 0:
        raise ScalifyError(status, where)


def scalify_matmul_scale_log2(K: int) -> int:
    return int(load_library().scalify_matmul_scale_log2(int(K)))


def scalify_mx_packed_bytes(rows: int, K: int) -> int:
    """Bytes of the packed form of an MX block-scale array (rows x K)."""
    return int(load_library().scalify_mx_packed_bytes(int(rows), int(K)))


def scalify_mx_pack_block_scales(src: torch.Tensor, K: int, stream=None) -> torch.Tensor:
    """Pack row-major E8M0 block-scale bytes src [rows, ld] (uint8 device
    tensor, ld >= ceil(K / 32), byte [r, k // 32] scaling row r's k) into the
    order scalify_matmul reads; returns a new uint8 device tensor."""
    if src.dtype != torch.uint8 or src.dim() != 2 or src.stride(1) != 1:
        raise ValueError("src: uint8 [rows, ld] with unit column stride")
    rows = src.shape[0]
    dst = torch.empty(max(scalify_mx_packed_bytes(rows, K), 4), dtype=torch.uint8,
                      device=src.device)
    st = load_library().scalify_mx_pack_block_scales(
        src.data_ptr() if src.numel() else None, rows, int(K), src.stride(0), dst.data_ptr(),
        _stream_handle(stream))
    _check(st, "scalify_mx_pack_block_scales")
    return dst[:scalify_mx_packed_bytes(rows, K)]


def scalify_matmul_workspace_size(M: int, N: int, out_fmt: int, rescale: int = RESCALE_AMAX) -> int:
    return int(load_library().scalify_matmul_workspace_size(M, N, out_fmt, rescale))


def scalify_matmul_workspace_size_opts(M: int, N: int, out_fmt: int, rescale: int = RESCALE_AMAX,
                                       fused: bool = False) -> int:
    """Workspace bytes of a call with (fused=True) or without a fused
    residual add, activation or pre_out export."""
    opts = CMatmulOpts(int(out_fmt), int(rescale), 0, 1, None, None, None, None, None,
                       ACT_RELU if fused else ACT_NONE, None)
    return int(load_library().scalify_matmul_workspace_size_opts(M, N, ctypes.byref(opts)))


def scalify_rescale_workspace_size(n: int) -> int:
    return int(load_library().scalify_rescale_workspace_size(n))


def workspace(nbytes: int, device) -> torch.Tensor:
    """Device workspace of nbytes, 256-byte aligned (torch allocations are)."""
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


def scalify_matmul(a: ScaledArray, b: ScaledArray, out: ScaledArray, *, rescale: int = RESCALE_AMAX,
                   target_log2: int = 0, saturate: bool = True, acc_out: torch.Tensor = None,
                   amax_out: torch.Tensor = None, amax_in: torch.Tensor = None,
                   residual: "ScaledArray" = None, activation: int = ACT_NONE,
                   pre_out: torch.Tensor = None, a_channel_scale: torch.Tensor = None,
                   b_channel_scale: torch.Tensor = None, a_block_scale: torch.Tensor = None,
                   b_block_scale: torch.Tensor = None,
                   ws: torch.Tensor = None, stream=None, events=None) -> None:
    """Scaled matmul (Section 3.2) with the fused dynamic or delayed rescale
    and cast (Section 3.3); see scalify_matmul in include/scalify.h.
    `amax_in` (RESCALE_DELAYED): one-element fp32 device tensor holding the
    statistic of an earlier call (its `amax_out`; may be the same tensor).
    `residual`: ScaledArray [M, N] added by the scaled add rule before the
    `activation` (ACT_*); a row broadcast as `bias.expand(M, N)` (stride 0)
    adds one row to every row. `pre_out`: fp32 [M, N] device tensor that
    receives the pre-cast value w (validation). `a_channel_scale` /
    `b_channel_scale`: contiguous fp32 device tensors [M] / [N] of powers of
    two, channel scales of a's rows / b's columns. `a_block_scale` /
    `b_block_scale`: MX block scales (E8M0, one per 32 k) of a's rows / b's
    columns, as returned by scalify_mx_pack_block_scales (uint8 device
    tensors of scalify_mx_packed_bytes(M or N, K) bytes).
    `events`: an optional sequence of 3 torch.cuda.Event(enable_timing=True)
    recorded before the GEMM kernel, after it and after the epilogue (None
    entries are skipped)."""
    lib = load_library()
    M, _ = a.shape
    _, N = b.shape
    opts, keep = _matmul_opts(a, out, rescale, target_log2, saturate, acc_out, amax_out, amax_in,
                              residual, activation, pre_out, a_channel_scale, b_channel_scale,
                              a_block_scale, b_block_scale, stream, events)
    if ws is None:
        ws = workspace(lib.scalify_matmul_workspace_size_opts(M, N, ctypes.byref(opts)),
                       a.data.device)
    ca, cb, co = a.c_struct(), b.c_struct(), out.c_struct()
    st = lib.scalify_matmul(ctypes.byref(ca), ctypes.byref(cb), ctypes.byref(co), ctypes.byref(opts),
                            ws.data_ptr(), ws.numel(), _stream_handle(stream))
    _check(st, "scalify_matmul")


def scalify_matmul_noalloc(a: ScaledArray, b: ScaledArray, out: ScaledArray, *,
                           rescale: int = RESCALE_AMAX, target_log2: int = 0,
                           saturate: bool = True, acc_out: torch.Tensor = None,
                           amax_out: torch.Tensor = None, amax_in: torch.Tensor = None,
                           residual: "ScaledArray" = None, activation: int = ACT_NONE,
                           pre_out: torch.Tensor = None, a_channel_scale: torch.Tensor = None,
                           b_channel_scale: torch.Tensor = None,
                           a_block_scale: torch.Tensor = None, b_block_scale: torch.Tensor = None,
                           stream=None, events=None) -> None:
    """scalify_matmul with the library's static workspace (no allocation by
    the library or by this binding); see scalify_matmul_noalloc in
    include/scalify.h for its size limit and its sharing rules."""
    lib = load_library()
    opts, keep = _matmul_opts(a, out, rescale, target_log2, saturate, acc_out, amax_out, amax_in,
                              residual, activation, pre_out, a_channel_scale, b_channel_scale,
                              a_block_scale, b_block_scale, stream, events)
    ca, cb, co = a.c_struct(), b.c_struct(), out.c_struct()
    st = lib.scalify_matmul_noalloc(ctypes.byref(ca), ctypes.byref(cb), ctypes.byref(co),
                                    ctypes.byref(opts), _stream_handle(stream))
    _check(st, "scalify_matmul_noalloc")


def _matmul_opts(a, out, rescale, target_log2, saturate, acc_out, amax_out, amax_in, residual,
                 activation, pre_out, a_channel_scale, b_channel_scale, a_block_scale,
                 b_block_scale, stream, events):
    """The scalify_matmul_opts struct of a call, and the ctypes objects it
    points to (kept alive by the caller until the call returns)."""
    M, K = a.shape
    N = out.shape[1]
    ev_arr = None
    if events is not None:
        for e in events:
            if e is not None and not e.cuda_event:       # torch creates its events lazily, on first record
                e.record(stream if stream is not None else torch.cuda.current_stream())
        ev_arr = (ctypes.c_void_p * 3)(*[e.cuda_event if e is not None else None for e in events])
    opts = CMatmulOpts(int(out.fmt), int(rescale), int(target_log2), int(bool(saturate)),
                       acc_out.data_ptr() if acc_out is not None else None,
                       amax_out.data_ptr() if amax_out is not None else None,
                       ctypes.cast(ev_arr, ctypes.c_void_p) if ev_arr is not None else None,
                       amax_in.data_ptr() if amax_in is not None else None,
                       None, int(activation), pre_out.data_ptr() if pre_out is not None else None,
                       a_channel_scale.data_ptr() if a_channel_scale is not None else None,
                       b_channel_scale.data_ptr() if b_channel_scale is not None else None,
                       a_block_scale.data_ptr() if a_block_scale is not None else None,
                       b_block_scale.data_ptr() if b_block_scale is not None else None)
    for t, rows in ((a_block_scale, M), (b_block_scale, N)):
        if t is not None and (t.dtype != torch.uint8 or not t.is_contiguous() or
                              t.numel() != scalify_mx_packed_bytes(rows, K)):
            raise ValueError("block scales: packed by scalify_mx_pack_block_scales")
    cr = residual.c_struct() if residual is not None else None
    if cr is not None:
        opts.residual = ctypes.pointer(cr)
    return opts, (ev_arr, cr)


def scalify_rescale(x: ScaledArray, out: ScaledArray, *, mode: int = RESCALE_AMAX, target_log2: int = 0,
                    saturate: bool = True, ws: torch.Tensor = None, stream=None) -> None:
    """Dynamic rescale (Section 3.3): amax -> power of two -> rebalance, plus cast."""
    lib = load_library()
    if ws is None:
        ws = workspace(scalify_rescale_workspace_size(x.data.numel()), x.data.device)
    ci, co = x.c_struct(), out.c_struct()
    st = lib.scalify_rescale(ctypes.byref(ci), ctypes.byref(co), int(mode), int(target_log2),
                             int(bool(saturate)), ws.data_ptr(), ws.numel(), _stream_handle(stream))
    _check(st, "scalify_rescale")


def scalify_cast(x: ScaledArray, out: ScaledArray, *, saturate: bool = True, stream=None) -> None:
    """Cast of the data component; the scale is copied (Appendix A)."""
    ci, co = x.c_struct(), out.c_struct()
    st = load_library().scalify_cast(ctypes.byref(ci), ctypes.byref(co), int(bool(saturate)),
                                     _stream_handle(stream))
    _check(st, "scalify_cast")


def scalify_set_scaling(x: ScaledArray, out: ScaledArray, new_scale_log2: int, *, saturate: bool = True,
                        stream=None) -> None:
    """set_scaling (Section 3.1): output scale 2^new_scale_log2, data rebalanced."""
    ci, co = x.c_struct(), out.c_struct()
    st = load_library().scalify_set_scaling(ctypes.byref(ci), ctypes.byref(co), int(new_scale_log2),
                                            int(bool(saturate)), _stream_handle(stream))
    _check(st, "scalify_set_scaling")


# ----------------------------------------------------------------------------- helpers

def _ptr_or_none(t: Optional[torch.Tensor]):
    return t.data_ptr() if t is not None else None


def scalify_layernorm_fwd(x: ScaledArray, out: ScaledArray, *, gamma: torch.Tensor = None,
                          beta: torch.Tensor = None, eps: float = 1e-5, saturate: bool = True,
                          pre_out: torch.Tensor = None, stream=None) -> None:
    """Scaled LayerNorm forward (Appendix C.2): normalizes x's data, output
    scale 1; see scalify_layernorm_fwd in include/scalify.h. gamma, beta:
    fp32 [D] device tensors or None."""
    lib = load_library()
    cx, co = x.c_struct(), out.c_struct()
    st = lib.scalify_layernorm_fwd(ctypes.byref(cx), _ptr_or_none(gamma), _ptr_or_none(beta),
                                   float(eps), ctypes.byref(co), int(bool(saturate)),
                                   _ptr_or_none(pre_out), _stream_handle(stream))
    _check(st, "scalify_layernorm_fwd")


def scalify_layernorm_bwd_workspace_size(R: int, D: int) -> int:
    return int(load_library().scalify_layernorm_bwd_workspace_size(R, D))


def scalify_layernorm_bwd(dy: ScaledArray, x: ScaledArray, dx: ScaledArray, *,
                          gamma: torch.Tensor = None, eps: float = 1e-5,
                          rescale: int = RESCALE_AMAX, target_log2: int = 0,
                          saturate: bool = True, dgamma: torch.Tensor = None,
                          dbeta: torch.Tensor = None, amax_out: torch.Tensor = None,
                          pre_out: torch.Tensor = None, ws: torch.Tensor = None,
                          stream=None) -> None:
    """LayerNorm input gradient with its dynamic rescale (Section 4, Section
    3.3); see scalify_layernorm_bwd in include/scalify.h."""
    lib = load_library()
    R, D = x.shape
    if ws is None:
        ws = workspace(scalify_layernorm_bwd_workspace_size(R, D), x.data.device)
    cdy, cx, cdx = dy.c_struct(), x.c_struct(), dx.c_struct()
    st = lib.scalify_layernorm_bwd(ctypes.byref(cdy), ctypes.byref(cx), _ptr_or_none(gamma),
                                   float(eps), ctypes.byref(cdx), _ptr_or_none(dgamma),
                                   _ptr_or_none(dbeta), int(rescale), int(target_log2),
                                   int(bool(saturate)), _ptr_or_none(amax_out),
                                   _ptr_or_none(pre_out), ws.data_ptr(), ws.numel(),
                                   _stream_handle(stream))
    _check(st, "scalify_layernorm_bwd")


def empty_scaled(rows: int, cols: int, fmt: int, device, ld: int = None) -> ScaledArray:
    """Output ScaledArray [rows, cols] with leading dimension ld (default: cols
    rounded up to 16 elements) and a fresh scale tensor."""
    if ld is None:
        ld = max(16, (cols + 15) // 16 * 16)
    storage = torch.empty((rows, ld), dtype=STORAGE_DTYPE[fmt], device=device)
    return ScaledArray(storage[:, :cols], fmt, torch.empty(1, dtype=torch.float32, device=device))


def scale_tensor(log2: int, device) -> torch.Tensor:
    return torch.tensor([2.0 ** log2], dtype=torch.float32, device=device)
