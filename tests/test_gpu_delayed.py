"""GPU parity of the delayed rescale of scalify_matmul (Section 3.3: the
rebalance uses the statistic an earlier call recorded, the call records its
own for the next one) through the C ABI, against the CPU oracle.

P1: codes, output scale and the recorded statistic equal the oracle's delayed
epilogue applied to the GPU's own accumulator (exact). The accumulator itself
is the same GEMM main loop as the dynamic mode (P2 in test_gpu_matmul.py);
one P2 check here covers the direct-cast epilogue's accumulator export.
"""
import itertools
import math

import numpy as np
import pytest
import torch

from oracle import oracle as orc
from paper_2407_17353_amd import binding as sc
from paper_2407_17353_amd import workloads as wl
from tests.helpers import check_p2_full, say, stored_with_padding

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _codes(shape, fmt, seed, heavy=False):
    return wl.fp8_normal(shape, fmt, seed, "cpu", 10.0 if heavy else None)


def _run(A_st, fa, ta, sa, B_st, fb, tb, sb, fout, amax_in, *, mode=sc.RESCALE_DELAYED,
         target=0, sat=True, stat=None, events=None):
    """One scalify_matmul call; `stat` (a device tensor) is used as both
    amax_in and amax_out when given, else a fresh tensor holding amax_in."""
    a = sc.ScaledArray(stored_with_padding(A_st, DEV), fa, sc.scale_tensor(sa, DEV), ta)
    b = sc.ScaledArray(stored_with_padding(B_st, DEV), fb, sc.scale_tensor(sb, DEV), tb)
    M, K = a.shape
    N = b.shape[1]
    out = sc.empty_scaled(M, N, fout, DEV)
    acc = torch.empty((M, N), dtype=torch.float32, device=DEV)
    if stat is None:
        stat_in = torch.tensor([amax_in], dtype=torch.float32, device=DEV)
        stat_out = torch.empty(1, dtype=torch.float32, device=DEV)
    else:
        stat_in = stat_out = stat
    sc.scalify_matmul(a, b, out, rescale=mode, target_log2=target, saturate=sat, acc_out=acc,
                      amax_out=stat_out, amax_in=stat_in if mode == sc.RESCALE_DELAYED else None)
    torch.cuda.synchronize()
    codes = out.data.cpu().numpy()
    if fout == sc.F16:
        codes = codes.view(np.uint16)
    s = float(out.scale.item())
    e_out = int(math.frexp(s)[1] - 1)
    assert s == 2.0 ** e_out
    return codes.copy(), e_out, float(stat_out.item()), acc.cpu().numpy(), K


def _check_p1(codes, e_out, amax, acc, K, sa, sb, fout, amax_in, target=0, sat=True):
    ref_codes, ref_e, ref_amax = orc.matmul_epilogue_delayed(acc, 2.0 ** sa, 2.0 ** sb, K, amax_in,
                                                             target, sat, fout)
    assert e_out == ref_e, (e_out, ref_e)
    assert np.float32(amax) == np.float32(ref_amax), (amax, ref_amax)
    bad = np.flatnonzero(codes.ravel() != ref_codes.ravel())
    assert bad.size == 0, f"P1: {bad.size} mismatches, first {bad[:5]} gpu " \
        f"{codes.ravel()[bad[:5]]} ref {ref_codes.ravel()[bad[:5]]} acc {acc.ravel()[bad[:5]]}"
    return ref_amax


SHAPES = [(1, 1, 1), (17, 33, 65), (257, 513, 129), (300, 200, 1000)]
LAYOUTS = list(itertools.product((False, True), repeat=2))


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("ta,tb", LAYOUTS, ids=lambda v: "T" if v else "N")
@pytest.mark.parametrize("fa,fb,fout", [(0, 0, 0), (1, 0, 1), (0, 1, 2), (1, 1, 0)],
                         ids=["e4m3-e4m3-e4m3", "e5m2-e4m3-e5m2", "e4m3-e5m2-f16", "e5m2-e5m2-e4m3"])
def test_delayed_p1_shapes_layouts_formats(shape, ta, tb, fa, fb, fout):
    M, N, K = shape
    say(f"case delayed {shape} ta={ta} tb={tb} fmts={fa},{fb}->{fout}")
    A = _codes((K, M) if ta else (M, K), fa, 300 + M, heavy=fa == sc.E5M2)
    B = _codes((N, K) if tb else (K, N), fb, 400 + N, heavy=fb == sc.E5M2)
    # statistics: one a call would have recorded on similar data, one far
    # too small (saturation), one far too large, and none yet
    for amax_in in (3.0, 2.0 ** -9, 2.0 ** 12, 0.0):
        codes, e_out, amax, acc, K_ = _run(A, fa, ta, -2, B, fb, tb, 1, fout, amax_in)
        _check_p1(codes, e_out, amax, acc, K_, -2, 1, fout, amax_in)


@pytest.mark.parametrize("fout", [sc.E4M3, sc.E5M2, sc.F16])
@pytest.mark.parametrize("target,sat", [(0, True), (0, False), (4, True)])
def test_delayed_targets_and_saturation(fout, target, sat):
    say(f"case delayed fout={fout} target={target} sat={sat}")
    A = _codes((200, 300), sc.E4M3, 51)
    B = _codes((300, 130), sc.E4M3, 52)
    for amax_in in (float("nan"), float("inf"), 1.0, 2.0 ** -20):
        codes, e_out, amax, acc, K = _run(A, sc.E4M3, False, 3, B, sc.E4M3, False, -4, fout,
                                          amax_in, target=target, sat=sat)
        _check_p1(codes, e_out, amax, acc, K, 3, -4, fout, amax_in, target, sat)


def test_delayed_with_the_current_statistic_equals_the_dynamic_rescale():
    """Fed the statistic this very product records, the delayed call gives
    the dynamic call's codes and scale bit for bit (same accumulator: P5)."""
    say("case delayed == dynamic")
    A = _codes((384, 1024), sc.E4M3, 61)
    B = _codes((1024, 640), sc.E4M3, 62)
    dyn = _run(A, sc.E4M3, False, 0, B, sc.E4M3, False, 2, sc.E4M3, 0.0, mode=sc.RESCALE_AMAX)
    dl = _run(A, sc.E4M3, False, 0, B, sc.E4M3, False, 2, sc.E4M3, dyn[2])
    assert np.array_equal(dyn[0], dl[0]) and dyn[1] == dl[1] and dyn[2] == dl[2]
    assert np.array_equal(dyn[3].view(np.uint32), dl[3].view(np.uint32))


def test_delayed_state_updated_in_place_across_calls():
    """amax_in and amax_out on one device word (the model state): the first
    call (no statistic yet) uses the static rule, the second the statistic
    the first recorded, which for the same product is the dynamic rescale."""
    say("case delayed chain")
    A = _codes((256, 512), sc.E4M3, 71)
    B = _codes((512, 320), sc.E4M3, 72)
    state = torch.zeros(1, dtype=torch.float32, device=DEV)
    first = _run(A, sc.E4M3, False, 0, B, sc.E4M3, False, 0, sc.E4M3, None, stat=state)
    _check_p1(first[0], first[1], first[2], first[3], first[4], 0, 0, sc.E4M3, 0.0)
    rec = float(state.item())
    second = _run(A, sc.E4M3, False, 0, B, sc.E4M3, False, 0, sc.E4M3, None, stat=state)
    _check_p1(second[0], second[1], second[2], second[3], second[4], 0, 0, sc.E4M3, rec)
    dyn = _run(A, sc.E4M3, False, 0, B, sc.E4M3, False, 0, sc.E4M3, 0.0, mode=sc.RESCALE_AMAX)
    assert np.array_equal(second[0], dyn[0]) and second[1] == dyn[1]


def test_delayed_accumulator_and_specials():
    """P2 of the exported accumulator, with NaN / Inf inputs (NaN excluded
    from the statistic, NaN codes keep their sign)."""
    say("case delayed specials")
    A = _codes((64, 256), sc.E5M2, 81).numpy().copy()
    B = _codes((256, 48), sc.E5M2, 82).numpy().copy()
    A[3, 7] = 0x7F
    A[9, 11] = 0x7C
    B[11, 2] = 0
    A_t, B_t = torch.from_numpy(A), torch.from_numpy(B)
    codes, e_out, amax, acc, K = _run(A_t, sc.E5M2, False, 0, B_t, sc.E5M2, False, 0, sc.E5M2, 8.0)
    _check_p1(codes, e_out, amax, acc, K, 0, 0, sc.E5M2, 8.0)
    check_p2_full(acc, A_t, sc.E5M2, False, B_t, sc.E5M2, False)
    assert np.isnan(acc[3]).all() and math.isinf(amax)


def test_delayed_empty_and_k_zero():
    say("case delayed empty")
    for M, N, K in [(0, 16, 16), (16, 0, 16), (16, 16, 0)]:
        A = torch.zeros((M, K), dtype=torch.uint8)
        B = torch.zeros((K, N), dtype=torch.uint8)
        a = sc.ScaledArray(A.to(DEV), sc.E4M3, sc.scale_tensor(2, DEV))
        b = sc.ScaledArray(B.to(DEV), sc.E4M3, sc.scale_tensor(3, DEV))
        out = sc.empty_scaled(M, N, sc.E4M3, DEV)
        out.data.fill_(0x55)
        st = torch.tensor([4.0], dtype=torch.float32, device=DEV)
        sc.scalify_matmul(a, b, out, rescale=sc.RESCALE_DELAYED, amax_in=st, amax_out=st)
        torch.cuda.synchronize()
        assert out.scale.item() == 2.0 ** (5 + sc.scalify_matmul_scale_log2(K) + 2)
        assert torch.all(out.data == 0).item()
        assert st.item() == 0.0


@pytest.mark.parametrize("size", [4096, 8192])
def test_delayed_square_full_size(size):
    """The square workload at full size, with the statistic of a previous
    call on other data of the same distribution (P1 on every element)."""
    case = wl.config_4(size, wl.E4M3)[0]
    say(f"case delayed {case.name}")
    A, B = case.make_a("cpu"), case.make_b("cpu")
    prev = _run(A[: size // 4], case.fa, False, case.a_scale_log2, B, case.fb, False,
                case.b_scale_log2, case.fout, 0.0, mode=sc.RESCALE_AMAX)
    codes, e_out, amax, acc, K = _run(A, case.fa, False, case.a_scale_log2, B, case.fb, False,
                                      case.b_scale_log2, case.fout, prev[2])
    _check_p1(codes, e_out, amax, acc, K, case.a_scale_log2, case.b_scale_log2, case.fout, prev[2])
    say(f"  P1 ok (statistic in {prev[2]:.4g}, recorded {amax:.4g})")


@pytest.mark.parametrize("fout", [sc.F16, sc.E4M3, sc.E5M2])
@pytest.mark.parametrize("amax_in,sat", [(2.0 ** -4, True), (2.0 ** -4, False), (2.0 ** 21, True),
                                         (2.0 ** 12, True)])
def test_delayed_integer_grid_rounding_boundaries(fout, amax_in, sat):
    """Integer-valued inputs (exact accumulators, K = 1000 -> e_c = 4):
    amax_in = 2^-4 casts the integers themselves (FP16 ties above 2048,
    overflow past 65504), 2^21 shifts them into the FP16 subnormals with
    ties at every odd value, 2^12 lands FP8 values on their ties."""
    say(f"case delayed grid fout={fout} amax_in={amax_in} sat={sat}")
    A = wl.int_grid((300, 1000), sc.E4M3, 91)
    B = wl.int_grid((1000, 260), sc.E4M3, 92)
    codes, e_out, amax, acc, K = _run(A, sc.E4M3, False, 0, B, sc.E4M3, False, 0, fout, amax_in,
                                      sat=sat)
    assert np.all(acc == np.round(acc))
    _check_p1(codes, e_out, amax, acc, K, 0, 0, fout, amax_in, 0, sat)
