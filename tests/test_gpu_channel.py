"""GPU parity of scalify_matmul with channel scales (a scale broadcastable
to the data, Section 2: one power of two per row of A and per column of B
on top of the scalar scales), through the C ABI, against the CPU oracle.

Each call exports its accumulator and pre-cast value w; the checks are the
fused epilogue's (tests/test_gpu_fused.py): F1 w against the oracle's value
from the GPU's own accumulator (bit for bit without a smooth gate), F2 the
codes, scale and statistic against the oracle's rescale and cast of the
GPU's w, and P2 of the accumulator.
"""
import itertools
import zlib

import numpy as np
import pytest

from paper_2407_17353_amd import binding as sc
from tests.helpers import check_p2_full, say
from tests.test_gpu_fused import _codes, _residual_codes, _run, check_fused

pytestmark = pytest.mark.gpu

LAYOUTS = list(itertools.product((False, True), repeat=2))
MODES = {"amax": sc.RESCALE_AMAX, "none": sc.RESCALE_NONE, "delayed": sc.RESCALE_DELAYED}


def _channels(M, N, seed, lo=-8, hi=8, which="both"):
    rng = np.random.default_rng(seed)
    ca = 2.0 ** rng.integers(lo, hi + 1, M) if which in ("both", "a") else None
    cb = 2.0 ** rng.integers(lo, hi + 1, N) if which in ("both", "b") else None
    return ca, cb


@pytest.mark.parametrize("mode", list(MODES))
@pytest.mark.parametrize("shape", [(1, 1, 1), (17, 33, 65), (257, 513, 129), (300, 200, 1000)],
                         ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("which", ["both", "a", "b"])
def test_channel_scales(which, shape, mode):
    M, N, K = shape
    i = zlib.crc32(f"{which}/{shape}/{mode}".encode()) % 1000  # stable across processes
    ta, tb = LAYOUTS[i % 4]
    fa, fb = [(0, 0), (1, 0), (0, 1), (1, 1)][(i // 4) % 4]
    fout = [sc.E4M3, sc.E5M2, sc.F16][i % 3]
    say(f"case channel {which} {shape} {mode} ta={ta} tb={tb} fmts={fa},{fb}->{fout}")
    A = _codes((M, K), fa, 700 + i, heavy=fa == 1)
    B = _codes((K, N), fb, 701 + i)
    A_st = A.t().contiguous() if ta else A
    B_st = B.t().contiguous() if tb else B
    ca, cb = _channels(M, N, i, which=which)
    run = _run(A_st, fa, ta, -1, B_st, fb, tb, 2, fout, mode=MODES[mode], amax_in=3.0,
               ch_a=ca, ch_b=cb)
    check_fused(run, -1, 2, fout, None, sc.ACT_NONE, MODES[mode], amax_in=3.0, ch_a=ca, ch_b=cb)
    check_p2_full(run[3], A_st, fa, ta, B_st, fb, tb)


@pytest.mark.parametrize("act", [sc.ACT_RELU, sc.ACT_GELU_TANH])
@pytest.mark.parametrize("rfmt", [None, sc.E4M3, sc.F16])
def test_channel_scales_with_residual_and_activation(rfmt, act):
    M, N, K = 130, 272, 384
    say(f"case channel res={rfmt} act={act}")
    A = _codes((M, K), sc.E4M3, 811)
    B = _codes((K, N), sc.E5M2, 812)
    ca, cb = _channels(M, N, 813, -5, 5)
    res = None if rfmt is None else (_residual_codes(M, N, rfmt, 814, spread=4), rfmt, 3)
    for mode in (sc.RESCALE_AMAX, sc.RESCALE_DELAYED):
        run = _run(A, sc.E4M3, False, 0, B, sc.E5M2, False, -3, sc.E4M3, res=res, act=act,
                   mode=mode, amax_in=0.5, ch_a=ca, ch_b=cb)
        check_fused(run, 0, -3, sc.E4M3, res, act, mode, amax_in=0.5, ch_a=ca, ch_b=cb)


def test_extreme_channel_exponents_saturate_and_flush_like_the_oracle():
    """Channel factors at the ends of the E8M0 range push w out of fp32's
    range (Inf) and into its subnormals: the kernel's power-of-two product
    must round and overflow exactly as the oracle's."""
    M, N, K = 64, 48, 256
    A = _codes((M, K), sc.E4M3, 821)
    B = _codes((K, N), sc.E4M3, 822)
    rng = np.random.default_rng(823)
    ca = 2.0 ** rng.choice([-127, -120, 0, 100, 127], M)
    cb = 2.0 ** rng.choice([-30, 0, 20], N)
    for sat in (True, False):
        run = _run(A, sc.E4M3, False, 0, B, sc.E4M3, False, 0, sc.F16, mode=sc.RESCALE_NONE,
                   sat=sat, ch_a=ca, ch_b=cb)
        check_fused(run, 0, 0, sc.F16, None, sc.ACT_NONE, sc.RESCALE_NONE, sat=sat, ch_a=ca, ch_b=cb)


def test_unit_channel_scales_match_the_plain_call():
    M, N, K = 200, 160, 512
    A = _codes((M, K), sc.E4M3, 831)
    B = _codes((K, N), sc.E4M3, 832)
    plain = _run(A, sc.E4M3, False, 1, B, sc.E4M3, False, -1, sc.E4M3)
    unit = _run(A, sc.E4M3, False, 1, B, sc.E4M3, False, -1, sc.E4M3, ch_a=np.ones(M),
                ch_b=np.ones(N))
    assert np.array_equal(plain[0], unit[0]) and plain[1:3] == unit[1:3]
    assert np.array_equal(plain[4].view(np.uint32), unit[4].view(np.uint32))


def test_channel_scale_alignment_is_checked():
    import torch
    M, N, K = 16, 32, 64
    A = _codes((M, K), sc.E4M3, 841)
    B = _codes((K, N), sc.E4M3, 842)
    cb = torch.ones(N + 1, dtype=torch.float32, device="cuda")[1:]  # 4-byte offset
    a = sc.ScaledArray(A.cuda(), sc.E4M3, sc.scale_tensor(0, "cuda"))
    b = sc.ScaledArray(B.cuda(), sc.E4M3, sc.scale_tensor(0, "cuda"))
    out = sc.empty_scaled(M, N, sc.E4M3, "cuda")
    with pytest.raises(sc.ScalifyError) as e:
        sc.scalify_matmul(a, b, out, b_channel_scale=cb)
    assert e.value.status == 5
