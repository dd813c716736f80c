"""GPU tests of the single-pass dynamic rescale and of the direct cast of the
persistent GEMM kernel (through the C ABI).

The single pass keeps each workgroup's last tile in its accumulators, meets
the other workgroups at a grid barrier on the amax statistic (Section 3.3),
casts that tile directly and its earlier tiles from the intermediate. AMAX
calls without a fused epilogue take it by default where every workgroup of
the persistent grid holds one tile; SCALIFY_SINGLE_PASS=1 forces it
wherever it can run, =0 never. It must give exactly the codes, scale and
statistic of the two-kernel path (GEMM + cast kernel), which the matmul
tests check against the oracle, and P1 against the oracle on the GPU's
accumulator. With a barrier
wait budget of 0 ticks (SCALIFY_SPIN_TICKS=0) a workgroup that is not the
last to arrive gives up at once: the kernel then takes its recovery path
(every held tile to the intermediate, the last workgroup to write casts
everything), which must give the same result; the barrier state word of the
workspace header records which path ran.

Calls without a rescale (NONE) and delayed calls cast in the GEMM epilogue
with a shift known before the GEMM; scales at the ends of the E8M0 range
push that shift outside the conversion's window (|shift| > 126), where the
values are scaled by v_ldexp first: P1 against the oracle there too.
"""
import contextlib
import math
import os

import numpy as np
import pytest
import torch

from oracle import oracle as orc
from paper_2407_17353_amd import binding as sc
from paper_2407_17353_amd import workloads as wl
from tests.helpers import check_p1, gpu_matmul, say, stored_with_padding

pytestmark = pytest.mark.gpu

DEV = "cuda"
HDR_STATE = 6  # workspace header word of the barrier state: 1 complete, 2 aborted


@contextlib.contextmanager
def env(**kw):
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


def _codes(shape, fmt, seed, heavy=False):
    return wl.fp8_normal(shape, fmt, seed, "cpu", 10.0 if heavy else None)


def run(A_st, fa, ta, sa, B_st, fb, tb, sb, fout, mode=sc.RESCALE_AMAX, want_acc=True):
    """scalify_matmul with a workspace of our own; returns (codes, e_out, amax,
    acc or None, barrier state word)."""
    a = sc.ScaledArray(stored_with_padding(A_st, DEV), fa, sc.scale_tensor(sa, DEV), ta)
    b = sc.ScaledArray(stored_with_padding(B_st, DEV), fb, sc.scale_tensor(sb, DEV), tb)
    M, K = a.shape
    _, N = b.shape
    out = sc.empty_scaled(M, N, fout, DEV)
    acc = torch.empty((M, N), dtype=torch.float32, device=DEV) if want_acc else None
    amax = torch.empty(1, dtype=torch.float32, device=DEV)
    ws = sc.workspace(sc.scalify_matmul_workspace_size(M, N, fout, mode), DEV)
    ws[:256].fill_(0xAB)  # the prologue must clear what the kernel relies on
    sc.scalify_matmul(a, b, out, rescale=mode, acc_out=acc, amax_out=amax, ws=ws)
    torch.cuda.synchronize()
    codes = out.data.cpu().numpy()
    if fout == sc.F16:
        codes = codes.view(np.uint16)
    s = float(out.scale.item())
    e_out = int(math.frexp(s)[1] - 1)
    assert s == 2.0 ** e_out
    state = int(ws[:32].cpu().view(torch.int32)[HDR_STATE].item())
    return (codes.copy(), e_out, float(amax.item()),
            acc.cpu().numpy() if want_acc else None, state)


# tiles of 256 x 256: 1 (one workgroup), 24 (one per workgroup, edges),
# 272 (more tiles than CUs: 16 workgroups hold a second tile), 512 (2 rounds)
SHAPES = [(200, 130, 300), (1024, 1500, 640), (4352, 4096, 256), (4096, 8192, 384)]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("fout", [sc.E4M3, sc.E5M2, sc.F16])
@pytest.mark.parametrize("want_acc", [False, True], ids=["noexport", "export"])
def test_single_pass_equals_two_kernel_path(shape, fout, want_acc):
    M, N, K = shape
    ta, tb = (M + N) % 2 == 1, (N // 2) % 2 == 1
    say(f"case single-pass M={M} N={N} K={K} ta={ta} tb={tb} fout={fout} export={want_acc}")
    A = _codes((M, K), sc.E4M3, 61 + M)
    B = _codes((K, N), sc.E5M2, 62 + N, heavy=True)
    A_st = A.t().contiguous() if ta else A
    B_st = B.t().contiguous() if tb else B
    with env(SCALIFY_SINGLE_PASS=1):
        r1 = run(A_st, sc.E4M3, ta, 2, B_st, sc.E5M2, tb, -3, fout, want_acc=want_acc)
    assert r1[4] == 1, "the barrier completed"
    with env(SCALIFY_SINGLE_PASS=0):
        r0 = run(A_st, sc.E4M3, ta, 2, B_st, sc.E5M2, tb, -3, fout, want_acc=want_acc)
    assert r0[4] == 0, "no barrier on the two-kernel path"
    assert np.array_equal(r0[0], r1[0]) and r0[1] == r1[1] and r0[2] == r1[2]
    # the default: the single pass exactly where no workgroup holds two tiles
    rd = run(A_st, sc.E4M3, ta, 2, B_st, sc.E5M2, tb, -3, fout, want_acc=False)
    tiles = -(-M // 256) * -(-N // 256)
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    assert rd[4] == (1 if tiles <= cus else 0)
    assert np.array_equal(rd[0], r1[0]) and rd[1] == r1[1] and rd[2] == r1[2]
    if want_acc:
        assert np.array_equal(r0[3].view(np.uint32), r1[3].view(np.uint32))
        check_p1(r1[0], r1[1], r1[2], r1[3], K, 2, -3, fout)


@pytest.mark.parametrize("shape", [(1024, 1500, 640), (4352, 4096, 256)],
                         ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("fout", [sc.E4M3, sc.F16])
def test_single_pass_abort_recovery(shape, fout):
    M, N, K = shape
    say(f"case single-pass abort M={M} N={N} K={K} fout={fout}")
    A = _codes((M, K), sc.E4M3, 71)
    B = _codes((K, N), sc.E4M3, 72)
    with env(SCALIFY_SINGLE_PASS=1):
        r1 = run(A, sc.E4M3, False, 0, B, sc.E4M3, False, 1, fout)
    assert r1[4] == 1
    with env(SCALIFY_SINGLE_PASS=1, SCALIFY_SPIN_TICKS=0):
        r2 = run(A, sc.E4M3, False, 0, B, sc.E4M3, False, 1, fout)
    assert r2[4] == 2, "the recovery path ran"
    assert np.array_equal(r1[0], r2[0]) and r1[1] == r2[1] and r1[2] == r2[2]
    check_p1(r2[0], r2[1], r2[2], r2[3], K, 0, 1, fout)


def test_single_pass_specials():
    """NaN / Inf accumulators through the single pass: NaN codes keep their
    sign, the Inf row dominates the statistic (no rescale)."""
    say("case single-pass specials")
    M, N, K = 300, 520, 256
    A = _codes((M, K), sc.E5M2, 81).numpy().copy()
    B = _codes((K, N), sc.E5M2, 82).numpy().copy()
    A[3, 7] = 0x7F   # NaN
    A[9, 11] = 0xFC  # -Inf
    A[290, 5] = 0xFF  # -NaN in the last row block
    At, Bt = torch.from_numpy(A), torch.from_numpy(B)
    for fout in (sc.E4M3, sc.E5M2, sc.F16):
        r = run(At, sc.E5M2, False, 0, Bt, sc.E5M2, False, 0, fout)
        check_p1(r[0], r[1], r[2], r[3], K, 0, 0, fout)
        assert math.isinf(r[2])


@pytest.mark.parametrize("mode", [sc.RESCALE_NONE, sc.RESCALE_AMAX])
@pytest.mark.parametrize("sa,sb", [(-127, -127), (127, 127), (-127, 120), (100, 27)])
@pytest.mark.parametrize("fout", [sc.E4M3, sc.E5M2, sc.F16])
def test_extreme_scales_outside_the_conversion_window(mode, sa, sb, fout):
    """Input scales at the E8M0 ends: the output scale clamps at 2^+-127, so
    the cast's shift leaves [-126, 126] (scaled by v_ldexp first) in NONE
    mode; P1 against the oracle on the GPU accumulator."""
    M, N, K = 300, 260, 200
    say(f"case extreme scales mode={mode} sa={sa} sb={sb} fout={fout}")
    A = _codes((M, K), sc.E4M3, 91)
    B = _codes((K, N), sc.E4M3, 92)
    codes, e_out, amax, acc = gpu_matmul(A, sc.E4M3, False, sa, B, sc.E4M3, False, sb, fout, mode)
    check_p1(codes, e_out, amax, acc, K, sa, sb, fout, mode)
    if mode == sc.RESCALE_NONE:
        e_c = sc.scalify_matmul_scale_log2(K)
        assert e_out == max(-127, min(127, sa + sb + e_c))


@pytest.mark.parametrize("fout", [sc.E4M3, sc.F16])
def test_none_mode_needs_no_intermediate(fout):
    """Without a rescale the output scale is known before the GEMM: the
    workspace is the header alone."""
    assert sc.scalify_matmul_workspace_size(8192, 8192, fout, sc.RESCALE_NONE) == 256
    M, N, K = 512, 768, 256
    A = _codes((M, K), sc.E4M3, 95)
    B = _codes((K, N), sc.E4M3, 96)
    a = sc.ScaledArray(A.to(DEV), sc.E4M3, sc.scale_tensor(-1, DEV))
    b = sc.ScaledArray(B.to(DEV), sc.E4M3, sc.scale_tensor(2, DEV))
    out = sc.empty_scaled(M, N, fout, DEV)
    acc = torch.empty((M, N), dtype=torch.float32, device=DEV)
    amax = torch.empty(1, dtype=torch.float32, device=DEV)
    sc.scalify_matmul(a, b, out, rescale=sc.RESCALE_NONE, acc_out=acc, amax_out=amax,
                      ws=sc.workspace(256, DEV))
    torch.cuda.synchronize()
    codes = out.data.cpu().numpy()
    if fout == sc.F16:
        codes = codes.view(np.uint16)
    e_out = int(math.frexp(float(out.scale.item()))[1] - 1)
    check_p1(codes, e_out, float(amax.item()), acc.cpu().numpy(), K, -1, 2, fout, sc.RESCALE_NONE)


def _direct(A_st, B_st, fmt, fout, mode, sat, want_acc, amax_in):
    a = sc.ScaledArray(stored_with_padding(A_st, DEV), fmt, sc.scale_tensor(1, DEV))
    b = sc.ScaledArray(stored_with_padding(B_st, DEV), fmt, sc.scale_tensor(-2, DEV))
    M, K = a.shape
    _, N = b.shape
    out = sc.empty_scaled(M, N, fout, DEV)
    acc = torch.empty((M, N), dtype=torch.float32, device=DEV) if want_acc else None
    amax = torch.empty(1, dtype=torch.float32, device=DEV)
    kw = {"amax_in": torch.tensor([amax_in], dtype=torch.float32, device=DEV)} \
        if mode == sc.RESCALE_DELAYED else {}
    sc.scalify_matmul(a, b, out, rescale=mode, saturate=sat, acc_out=acc, amax_out=amax, **kw)
    torch.cuda.synchronize()
    codes = out.data.cpu().numpy()
    if fout == sc.F16:
        codes = codes.view(np.uint16)
    return (codes.copy(), float(out.scale.item()), float(amax.item()),
            acc.cpu().numpy() if want_acc else None)


@pytest.mark.parametrize("mode", [sc.RESCALE_NONE, sc.RESCALE_DELAYED])
@pytest.mark.parametrize("fout", [sc.E4M3, sc.E5M2, sc.F16])
@pytest.mark.parametrize("sat", [True, False], ids=["sat", "nosat"])
def test_direct_cast_interior_path_equals_the_checked_path(mode, fout, sat):
    """The direct cast of a wave tile inside the matrix (shift inside the
    conversion window, no exported accumulator: saturation chosen per tile,
    NaN groups on their own branch, FP16 through a clamp) gives the codes,
    scale and statistic of the per-element path that the same call takes
    when it exports its accumulators, which P1 checks against the oracle.
    Heavy-range E5M2 inputs overflow the output formats; NaN and Inf
    accumulators sit in interior wave tiles."""
    say(f"case direct interior mode={mode} fout={fout} sat={sat}")
    M, N, K = 512, 384, 256
    A = _codes((M, K), sc.E5M2, 131, heavy=True).numpy().copy()
    B = _codes((K, N), sc.E5M2, 132, heavy=True).numpy().copy()
    A[3, 7] = 0x7F     # NaN row
    A[9, 11] = 0x7C    # +Inf row ...
    B[11, 2] = 0       # ... with Inf * 0 = NaN at (9, 2)
    A[140, 5] = 0xFF   # -NaN row
    A[260, 9] = 0xFC   # -Inf row
    At, Bt = torch.from_numpy(A), torch.from_numpy(B)
    stat = 3.0e4  # the delayed statistic: a shift inside the window
    fast = _direct(At, Bt, sc.E5M2, fout, mode, sat, False, stat)
    ref = _direct(At, Bt, sc.E5M2, fout, mode, sat, True, stat)
    assert np.array_equal(fast[0], ref[0]), \
        f"{np.count_nonzero(fast[0] != ref[0])} codes differ"
    assert fast[1] == ref[1] and np.float32(fast[2]) == np.float32(ref[2])
    e_out = int(math.frexp(ref[1])[1] - 1)
    if mode == sc.RESCALE_NONE:
        check_p1(ref[0], e_out, ref[2], ref[3], K, 1, -2, fout, mode, saturate=sat)
    assert np.isnan(ref[3][3]).all() and np.isnan(ref[3][9, 2]) and np.isnan(ref[3][140]).all()


@pytest.mark.parametrize("single_pass", [0, 1], ids=["pair", "single"])
@pytest.mark.parametrize("fout", [sc.E4M3, sc.E5M2, sc.F16])
@pytest.mark.parametrize("sat", [True, False], ids=["sat", "nosat"])
def test_dynamic_rescale_interior_path_equals_the_checked_path(single_pass, fout, sat):
    """The dynamic rescale without an exported accumulator (interior wave
    tiles stored without per-element checks, or held by the single pass)
    gives the codes, scale and statistic of the same call with the export,
    which P1 checks against the oracle."""
    say(f"case dynamic interior single_pass={single_pass} fout={fout} sat={sat}")
    M, N, K = 512, 384, 256
    A = _codes((M, K), sc.E5M2, 141, heavy=True).numpy().copy()
    B = _codes((K, N), sc.E5M2, 142, heavy=True).numpy().copy()
    A[3, 7] = 0x7F
    A[140, 5] = 0xFF
    At, Bt = torch.from_numpy(A), torch.from_numpy(B)
    with env(SCALIFY_SINGLE_PASS=single_pass):
        fast = gpu_matmul(At, sc.E5M2, False, 1, Bt, sc.E5M2, False, -2, fout, saturate=sat,
                          want_acc=False)
        ref = gpu_matmul(At, sc.E5M2, False, 1, Bt, sc.E5M2, False, -2, fout, saturate=sat)
    assert np.array_equal(fast[0], ref[0]), f"{np.count_nonzero(fast[0] != ref[0])} codes differ"
    assert fast[1] == ref[1] and np.float32(fast[2]) == np.float32(ref[2])
    check_p1(ref[0], ref[1], ref[2], ref[3], K, 1, -2, fout, saturate=sat)
