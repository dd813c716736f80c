"""Seeded synthetic inputs for the scaled-matmul workloads.

This module holds no arithmetic of the method: it draws random numbers with
torch generators and encodes them to FP8 codes with torch's own float8
conversion (a library routine), so that the HIP path and the CPU oracle can
be fed identical bytes. Shapes and distributions follow the benchmark
configurations:

  1  single matmul 256^3, E4M3 N(0,1) data, scales 2^-3 and 2^5, E4M3 out
  2  Transformer MLP forward, d_model 2048, d_ff 8192, 4096 tokens, E4M3
  3  backward of that MLP: E5M2 gradients N(0,1) * 2^U(-10,0) per row
  4  square sweep 4096 / 8192 / 16384, E4M3 inputs, scales 2^U{-8..8},
     FP16 and E4M3 outputs
  5  LLaMA-7B-shaped layer GEMMs, 16384 tokens, d 4096, QKV 12288, MLP
     11008, forward E4M3 and backward E5M2 gradients

Seeds: 240717353 + 100 * config + tensor index.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Callable, Dict, List, Optional

import torch

E4M3, E5M2, F16 = 0, 1, 2
RESCALE_NONE, RESCALE_AMAX = 0, 1
_TORCH_FP8 = {E4M3: torch.float8_e4m3fn, E5M2: torch.float8_e5m2}
BASE_SEED = 240717353


def seed_of(cfg: int, idx: int) -> int:
    return BASE_SEED + 100 * cfg + idx


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def fp8_normal(shape, fmt: int, seed: int, device="cpu", row_log2_range: Optional[float] = None):
    """FP8 codes (uint8) of N(0,1) samples; with row_log2_range = r, row i is
    multiplied by 2^u_i, u_i ~ U(-r, 0) (heavy dynamic range across rows)."""
    g = _gen(seed, device)
    x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if row_log2_range is not None:
        u = torch.rand((shape[0], 1), generator=g, device=device, dtype=torch.float32)
        x = x * torch.exp2(-row_log2_range * u)
    return x.to(_TORCH_FP8[fmt]).view(torch.uint8)


def int_grid(shape, fmt: int, seed: int, device="cpu", vmax: int = 8):
    """FP8 codes whose values are integers in [-vmax, vmax] (every partial sum
    is exact in fp32 at the benchmark sizes)."""
    g = _gen(seed, device)
    v = torch.randint(-vmax, vmax + 1, shape, generator=g, device=device).to(torch.float32)
    return v.to(_TORCH_FP8[fmt]).view(torch.uint8)


def mx_block_scales(rows: int, K: int, seed: int, lo: int = -8, hi: int = 8, device="cpu"):
    """Row-major E8M0 block-scale bytes [rows][4 * ceil(K / 128)] (one per 32 k,
    padded to whole 128-k steps): 127 + an exponent uniform in [lo, hi], the
    spread of per-block scales of FP8 data quantized block by block."""
    ld = 4 * ((K + 127) // 128)
    e = torch.randint(lo, hi + 1, (rows, ld), generator=_gen(seed, "cpu"), dtype=torch.int32)
    return (e + 127).to(torch.uint8).to(device)


def scale_log2_draw(seed: int, lo: int, hi: int) -> int:
    g = _gen(seed, "cpu")
    return int(torch.randint(lo, hi + 1, (1,), generator=g).item())


@dataclass
class GemmCase:
    """One scaled GEMM: logical A [M,K] times B [K,N]. A is stored [K][M]
    when ta, B is stored [N][K] when tb. make_a / make_b build the stored
    code matrices on a device."""
    name: str
    M: int
    N: int
    K: int
    fa: int
    fb: int
    fout: int
    ta: bool
    tb: bool
    a_scale_log2: int
    b_scale_log2: int
    make_a: Callable = field(repr=False, default=None)
    make_b: Callable = field(repr=False, default=None)
    mode: int = RESCALE_AMAX

    @property
    def flops(self) -> int:
        return 2 * self.M * self.N * self.K

    def a_stored_shape(self):
        return (self.K, self.M) if self.ta else (self.M, self.K)

    def b_stored_shape(self):
        return (self.N, self.K) if self.tb else (self.K, self.N)


def _normal_maker(shape, fmt, seed, heavy=False):
    return lambda device: fp8_normal(shape, fmt, seed, device, 10.0 if heavy else None)


def config_1() -> List[GemmCase]:
    s = (256, 256)
    return [GemmCase("cfg1_256", 256, 256, 256, E4M3, E4M3, E4M3, False, False, -3, 5,
                     _normal_maker(s, E4M3, seed_of(1, 0)), _normal_maker(s, E4M3, seed_of(1, 1)))]


def _mlp_weights_scales(cfg: int):
    return scale_log2_draw(seed_of(cfg, 50), -6, -4), scale_log2_draw(seed_of(cfg, 51), -6, -4)


def config_2() -> List[GemmCase]:
    T, d, f = 4096, 2048, 8192
    s1, s2 = _mlp_weights_scales(2)
    X = _normal_maker((T, d), E4M3, seed_of(2, 0))
    W1 = _normal_maker((d, f), E4M3, seed_of(2, 1))
    W2 = _normal_maker((f, d), E4M3, seed_of(2, 2))
    H = _normal_maker((T, f), E4M3, seed_of(2, 3))   # stands in for the rescaled H when run alone
    return [GemmCase("cfg2_fwd_h", T, f, d, E4M3, E4M3, E4M3, False, False, 0, s1, X, W1),
            GemmCase("cfg2_fwd_y", T, d, f, E4M3, E4M3, E4M3, False, False, 0, s2, H, W2)]


def config_3() -> List[GemmCase]:
    T, d, f = 4096, 2048, 8192
    s1, s2 = _mlp_weights_scales(2)      # the same weights as the forward
    X = _normal_maker((T, d), E4M3, seed_of(2, 0))
    W1 = _normal_maker((d, f), E4M3, seed_of(2, 1))
    W2 = _normal_maker((f, d), E4M3, seed_of(2, 2))
    H = _normal_maker((T, f), E4M3, seed_of(2, 3))
    dY = _normal_maker((T, d), E5M2, seed_of(3, 0), heavy=True)
    dH = _normal_maker((T, f), E5M2, seed_of(3, 1), heavy=True)  # stands in for the rescaled dH
    return [GemmCase("cfg3_dh", T, f, d, E5M2, E4M3, E5M2, False, True, 0, s2, dY, W2),
            GemmCase("cfg3_dw2", f, d, T, E4M3, E5M2, E5M2, True, False, 0, 0, H, dY),
            GemmCase("cfg3_dx", T, d, f, E5M2, E4M3, E5M2, False, True, 0, s1, dH, W1),
            GemmCase("cfg3_dw1", d, f, T, E4M3, E5M2, E5M2, True, False, 0, 0, X, dH)]


def config_4(size: int, fout: int = E4M3) -> List[GemmCase]:
    sa = scale_log2_draw(seed_of(4, 10 + size % 97), -8, 8)
    sb = scale_log2_draw(seed_of(4, 20 + size % 97), -8, 8)
    A = _normal_maker((size, size), E4M3, seed_of(4, 0))
    B = _normal_maker((size, size), E4M3, seed_of(4, 1))
    tag = {E4M3: "e4m3", F16: "f16"}[fout]
    return [GemmCase(f"cfg4_sq{size}_{tag}", size, size, size, E4M3, E4M3, fout, False, False,
                     sa, sb, A, B)]


def config_5() -> List[GemmCase]:
    T, d, q, f = 16384, 4096, 12288, 11008
    ws = [scale_log2_draw(seed_of(5, 50 + i), -6, -4) for i in range(4)]
    X = _normal_maker((T, d), E4M3, seed_of(5, 0))
    O = _normal_maker((T, d), E4M3, seed_of(5, 1))
    Hn = _normal_maker((T, d), E4M3, seed_of(5, 2))
    U = _normal_maker((T, f), E4M3, seed_of(5, 3))
    Wqkv = _normal_maker((d, q), E4M3, seed_of(5, 4))
    Wo = _normal_maker((d, d), E4M3, seed_of(5, 5))
    Wup = _normal_maker((d, f), E4M3, seed_of(5, 6))
    Wdn = _normal_maker((f, d), E4M3, seed_of(5, 7))
    dQKV = _normal_maker((T, q), E5M2, seed_of(5, 8), heavy=True)
    dO = _normal_maker((T, d), E5M2, seed_of(5, 9), heavy=True)
    dUp = _normal_maker((T, f), E5M2, seed_of(5, 10), heavy=True)
    dDn = _normal_maker((T, d), E5M2, seed_of(5, 11), heavy=True)
    cases = []
    for name, act, W, dOut, n_in, n_out, sw in (("qkv", X, Wqkv, dQKV, d, q, ws[0]),
                                                ("attn_out", O, Wo, dO, d, d, ws[1]),
                                                ("mlp_up", Hn, Wup, dUp, d, f, ws[2]),
                                                ("mlp_down", U, Wdn, dDn, f, d, ws[3])):
        cases.append(GemmCase(f"cfg5_{name}_fwd", T, n_out, n_in, E4M3, E4M3, E4M3, False, False,
                              0, sw, act, W))
        cases.append(GemmCase(f"cfg5_{name}_dx", T, n_in, n_out, E5M2, E4M3, E5M2, False, True,
                              0, sw, dOut, W))
        cases.append(GemmCase(f"cfg5_{name}_dw", n_in, n_out, T, E4M3, E5M2, E5M2, True, False,
                              0, 0, act, dOut))
    return cases


def all_configs() -> Dict[int, List[GemmCase]]:
    return {1: config_1(), 2: config_2(), 3: config_3(),
            4: config_4(4096) + config_4(4096, F16) + config_4(8192) + config_4(8192, F16)
            + config_4(16384) + config_4(16384, F16),
            5: config_5()}
