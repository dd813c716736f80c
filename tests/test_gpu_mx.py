"""GPU parity of scalify_matmul with MX block scales (Section 2: a scale
broadcastable to the data covers block-scaling formats such as MX: one
E8M0 byte per 32 consecutive k of each row of A and column of B, applied by
the matrix cores' scaled MFMA), through the C ABI, against the CPU oracle.

P2: the exported accumulator against the oracle's block-scaled sum, within
the fp32 accumulation tolerance of the l1 norm of the scaled product terms.
P1: codes, output scale and statistic equal the oracle epilogue's on the
GPU's own accumulator, bit for bit. Cross-checks: all bytes 127 reproduce
the plain call bit for bit; bytes constant along k reproduce the channel-
scale call; padding bytes are never used.
"""
import itertools
import math
import zlib

import numpy as np
import pytest
import torch

from oracle import oracle as orc
from paper_2407_17353_amd import binding as sc
from paper_2407_17353_amd import workloads as wl
from tests.helpers import FMT, _compare_acc, check_p1, record, say, stored_with_padding

pytestmark = pytest.mark.gpu
DEV = "cuda"
LAYOUTS = list(itertools.product((False, True), repeat=2))
MODES = {"amax": sc.RESCALE_AMAX, "none": sc.RESCALE_NONE, "delayed": sc.RESCALE_DELAYED}


def _codes(shape, fmt, seed):
    return wl.fp8_normal(shape, fmt, seed, "cpu")


def _mx_run(A_st, fa, ta, sa, B_st, fb, tb, sb, fout, PA, PB, mode=sc.RESCALE_AMAX,
            amax_in=0.0, sat=True, want_acc=True):
    """One scalify_matmul call with block scales PA [M, ld], PB [N, ld]
    (uint8 tensors; None = a plain call). Returns codes, e_out, amax, acc."""
    a = sc.ScaledArray(stored_with_padding(A_st, DEV), fa, sc.scale_tensor(sa, DEV), ta)
    b = sc.ScaledArray(stored_with_padding(B_st, DEV), fb, sc.scale_tensor(sb, DEV), tb)
    M, K = a.shape
    N = b.shape[1]
    out = sc.empty_scaled(M, N, fout, DEV)
    acc = torch.empty((M, N), dtype=torch.float32, device=DEV) if want_acc else None
    stat_in = torch.tensor([amax_in], dtype=torch.float32, device=DEV)
    stat_out = torch.empty(1, dtype=torch.float32, device=DEV)
    pa = None if PA is None else sc.scalify_mx_pack_block_scales(PA.to(DEV), K)
    pb = None if PB is None else sc.scalify_mx_pack_block_scales(PB.to(DEV), K)
    sc.scalify_matmul(a, b, out, rescale=mode, saturate=sat, acc_out=acc, amax_out=stat_out,
                      amax_in=stat_in if mode == sc.RESCALE_DELAYED else None,
                      a_block_scale=pa, b_block_scale=pb)
    torch.cuda.synchronize()
    codes = out.data.cpu().numpy()
    if fout == sc.F16:
        codes = codes.view(np.uint16)
    s = float(out.scale.item())
    e_out = int(math.frexp(s)[1] - 1)
    assert s == 2.0 ** e_out
    return codes.copy(), e_out, float(stat_out.item()), (acc.cpu().numpy() if want_acc else None)


def _check(run, A_st, fa, ta, sa, B_st, fb, tb, sb, fout, PA, PB, mode, amax_in=0.0, sat=True):
    codes, e_out, amax, acc = run
    A, B = A_st.numpy(), B_st.numpy()
    K = A.shape[0] if ta else A.shape[1]
    pa, pb = PA.numpy(), PB.numpy()
    ref = orc.matmul_acc_mx(A, fa, ta, B, fb, tb, pa, pb)
    l1 = orc.matmul_acc_mx(A & 0x7F, fa, ta, B & 0x7F, fb, tb, pa, pb)  # |value| codes
    _compare_acc(acc, ref, l1.astype(np.float64), K)                     # P2
    if mode == sc.RESCALE_DELAYED:                                        # P1
        rc, re, ra = orc.matmul_epilogue_delayed(acc, 2.0 ** sa, 2.0 ** sb, K, amax_in, 0, sat, fout)
        assert e_out == re and np.float32(amax) == np.float32(ra), (e_out, re, amax, ra)
        bad = np.flatnonzero(codes.ravel() != rc.ravel())
        assert bad.size == 0, f"P1: {bad.size} code mismatches, first {bad[:5]}"
    else:
        check_p1(codes, e_out, amax, acc, K, sa, sb, fout, mode, saturate=sat)


@pytest.mark.parametrize("mode", list(MODES))
@pytest.mark.parametrize("shape", [(1, 1, 1), (17, 33, 65), (257, 513, 129), (300, 200, 1000),
                                   (130, 272, 4096)], ids=lambda s: "x".join(map(str, s)))
def test_block_scales(shape, mode):
    M, N, K = shape
    i = zlib.crc32(f"{shape}/{mode}".encode()) % 1000  # stable across processes
    ta, tb = LAYOUTS[i % 4]
    fa, fb = [(0, 0), (1, 0), (0, 1), (1, 1)][(i // 4) % 4]
    fout = [sc.E4M3, sc.E5M2, sc.F16][i % 3]
    say(f"case mx {shape} {mode} ta={ta} tb={tb} fmts={fa},{fb}->{fout}")
    A = _codes((M, K), fa, 900 + i)
    B = _codes((K, N), fb, 901 + i)
    A_st = A.t().contiguous() if ta else A
    B_st = B.t().contiguous() if tb else B
    PA = wl.mx_block_scales(M, K, 902 + i)
    PB = wl.mx_block_scales(N, K, 903 + i)
    run = _mx_run(A_st, fa, ta, -1, B_st, fb, tb, 2, fout, PA, PB, MODES[mode], amax_in=3.0)
    _check(run, A_st, fa, ta, -1, B_st, fb, tb, 2, fout, PA, PB, MODES[mode], amax_in=3.0)


@pytest.mark.parametrize("ta,tb", LAYOUTS, ids=lambda v: "T" if v else "N")
def test_wide_exponent_spread_every_layout(ta, tb):
    """Per-block exponents over [-40, 40]: block sums of very different
    magnitudes in one accumulator, both formats mixed, saturating and not."""
    M, N, K = 192, 320, 1024 + 96
    say(f"case mx wide ta={ta} tb={tb}")
    A = _codes((M, K), sc.E5M2, 911)
    B = _codes((K, N), sc.E4M3, 912)
    A_st = A.t().contiguous() if ta else A
    B_st = B.t().contiguous() if tb else B
    PA = wl.mx_block_scales(M, K, 913, -40, 40)
    PB = wl.mx_block_scales(N, K, 914, -40, 40)
    for sat in (True, False):
        run = _mx_run(A_st, sc.E5M2, ta, 0, B_st, sc.E4M3, tb, 0, sc.E4M3, PA, PB, sat=sat)
        _check(run, A_st, sc.E5M2, ta, 0, B_st, sc.E4M3, tb, 0, sc.E4M3, PA, PB, sc.RESCALE_AMAX,
               sat=sat)


@pytest.mark.parametrize("shape", [(200, 160, 512), (300, 520, 1000), (1024, 256, 4096)],
                         ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("mode", [sc.RESCALE_AMAX, sc.RESCALE_DELAYED])
def test_unit_block_scales_match_the_plain_call(shape, mode):
    """Bytes 127 (factor 1): the oracle's unscaled parity, and the plain
    call's accumulator within fp32 accumulation rounding. (Not bit for bit:
    the block-scaled kernels hand each MFMA its k in the matrix cores' own
    order, the plain ones in another; the products each MFMA sums, and so
    the rounding of its partial sums, differ.)"""
    M, N, K = shape
    say(f"case mx unit {shape} mode={mode}")
    A = _codes((M, K), sc.E4M3, 921)
    B = _codes((K, N), sc.E5M2, 922)
    ld = orc.mx_block_scale_ld(K)
    PA = torch.full((M, ld), 127, dtype=torch.uint8)
    PB = torch.full((N, ld), 127, dtype=torch.uint8)
    plain = _mx_run(A, sc.E4M3, False, 1, B, sc.E5M2, False, -1, sc.E4M3, None, None, mode, 2.0)
    unit = _mx_run(A, sc.E4M3, False, 1, B, sc.E5M2, False, -1, sc.E4M3, PA, PB, mode, 2.0)
    _check(unit, A, sc.E4M3, False, 1, B, sc.E5M2, False, -1, sc.E4M3, PA, PB, mode, amax_in=2.0)
    l1 = orc.matmul_acc(A.numpy() & 0x7F, sc.E4M3, False, B.numpy() & 0x7F, sc.E5M2, False)
    diff = np.abs(plain[3].astype(np.float64) - unit[3])
    assert np.all(diff <= 2.0 ** -20 * l1), float((diff / np.maximum(l1, 1e-30)).max())


def test_bytes_constant_along_k_match_channel_scales():
    """A byte constant along k is a channel factor: oracle parity, and the
    accumulator within fp32 accumulation rounding of the channel-scale
    call's pre-cast value w (another kernel and epilogue path), with the
    same output scale."""
    M, N, K = 260, 300, 768
    say("case mx vs channel")
    A = _codes((M, K), sc.E4M3, 931)
    B = _codes((K, N), sc.E4M3, 932)
    rng = np.random.default_rng(933)
    ca, cb = rng.integers(-12, 13, M), rng.integers(-12, 13, N)
    ld = orc.mx_block_scale_ld(K)
    PA = torch.from_numpy(np.repeat((127 + ca)[:, None], ld, axis=1).astype(np.uint8))
    PB = torch.from_numpy(np.repeat((127 + cb)[:, None], ld, axis=1).astype(np.uint8))
    mx = _mx_run(A, sc.E4M3, False, 0, B, sc.E4M3, False, 0, sc.E4M3, PA, PB)
    a = sc.ScaledArray(stored_with_padding(A, DEV), sc.E4M3, sc.scale_tensor(0, DEV), False)
    b = sc.ScaledArray(stored_with_padding(B, DEV), sc.E4M3, sc.scale_tensor(0, DEV), False)
    out = sc.empty_scaled(M, N, sc.E4M3, DEV)
    pre = torch.empty((M, N), dtype=torch.float32, device=DEV)
    stat = torch.empty(1, dtype=torch.float32, device=DEV)
    sc.scalify_matmul(a, b, out, amax_out=stat, pre_out=pre,
                      a_channel_scale=torch.exp2(torch.from_numpy(ca).float()).to(DEV),
                      b_channel_scale=torch.exp2(torch.from_numpy(cb).float()).to(DEV))
    torch.cuda.synchronize()
    _check(mx, A, sc.E4M3, False, 0, B, sc.E4M3, False, 0, sc.E4M3, PA, PB, sc.RESCALE_AMAX)
    l1 = orc.matmul_acc_mx(A.numpy() & 0x7F, sc.E4M3, False, B.numpy() & 0x7F, sc.E4M3, False,
                           PA.numpy(), PB.numpy())
    diff = np.abs(mx[3].astype(np.float64) - pre.cpu().numpy())
    assert np.all(diff <= 2.0 ** -20 * l1), float((diff / np.maximum(l1, 1e-30)).max())
    assert mx[1] == int(math.frexp(float(out.scale.item()))[1] - 1)
    assert abs(mx[2] - float(stat.item())) <= 2.0 ** -18 * abs(mx[2])


def test_padding_bytes_are_not_used():
    """K = 200 uses 7 of the 8 bytes of a row: an 0xFF (NaN) or 0 byte in
    the eighth changes nothing; nor do rows past a partial tile."""
    M, N, K = 70, 90, 200
    say("case mx padding")
    A = _codes((M, K), sc.E4M3, 941)
    B = _codes((K, N), sc.E4M3, 942)
    PA = wl.mx_block_scales(M, K, 943)
    PB = wl.mx_block_scales(N, K, 944)
    PA[:, 7] = 127
    PB[:, 7] = 127
    r0 = _mx_run(A, sc.E4M3, False, 0, B, sc.E4M3, False, 0, sc.E5M2, PA, PB)
    PA2, PB2 = PA.clone(), PB.clone()
    PA2[:, 7] = 0xFF
    PB2[:, 7] = 0
    r1 = _mx_run(A, sc.E4M3, False, 0, B, sc.E4M3, False, 0, sc.E5M2, PA2, PB2)
    assert np.array_equal(r0[3].view(np.uint32), r1[3].view(np.uint32))
    assert np.array_equal(r0[0], r1[0]) and r0[1:3] == r1[1:3]
    _check(r1, A, sc.E4M3, False, 0, B, sc.E4M3, False, 0, sc.E5M2, PA2, PB2, sc.RESCALE_AMAX)


@pytest.mark.parametrize("rows,K", [(1, 1), (17, 65), (64, 128), (300, 1000), (130, 4096 + 32)])
def test_pack_order(rows, K):
    """The packed order written out independently with numpy: word
    ((t * G + q) * 64 + 16 g + r) holds rows 64 q + r + 16 i (byte i) at
    k-block 4 t + g, with 127 outside the array."""
    say(f"case mx pack {rows}x{K}")
    src = wl.mx_block_scales(rows, K, 961)
    got = sc.scalify_mx_pack_block_scales(src.to(DEV), K).cpu().numpy()
    nb, T, G = (K + 31) // 32, (K + 127) // 128, (rows + 63) // 64
    full = np.full((G * 64, 4 * T), 127, np.uint8)
    full[:rows, :nb] = src.numpy()[:, :nb]
    want = full.reshape(G, 4, 16, T, 4)            # [q][i][r][t][g]
    want = want.transpose(3, 0, 4, 2, 1).reshape(-1)  # [t][q][g][r][i]
    assert got.size == sc.scalify_mx_packed_bytes(rows, K) == want.size
    assert np.array_equal(got, want)


def test_empty_and_zero_depth():
    for M, N, K in ((0, 16, 64), (16, 0, 64), (16, 16, 0)):
        say(f"case mx empty {M}x{N}x{K}")
        A = torch.zeros((M, K), dtype=torch.uint8)
        B = torch.zeros((K, N), dtype=torch.uint8)
        ld = orc.mx_block_scale_ld(K)
        PA = torch.full((M, ld), 127, dtype=torch.uint8)
        PB = torch.full((N, ld), 127, dtype=torch.uint8)
        codes, e_out, amax, acc = _mx_run(A, 0, False, 0, B, 0, False, 0, sc.E4M3, PA, PB)
        assert codes.shape == (M, N) and not codes.any() and not acc.any()
        assert amax == 0.0


def test_headline_shape_sampled():
    """8192^3 E4M3 with block scales (the benchmark's block-scale line): P2
    on sampled outputs summed by the oracle one by one, P1 on every code."""
    case = wl.config_4(8192, sc.E4M3)[0]
    say(f"case mx headline {case.name}")
    A, B = case.make_a("cpu"), case.make_b("cpu")
    PA = wl.mx_block_scales(case.M, case.K, 951)
    PB = wl.mx_block_scales(case.N, case.K, 952)
    codes, e_out, amax, acc = _mx_run(A, case.fa, case.ta, case.a_scale_log2, B, case.fb, case.tb,
                                      case.b_scale_log2, case.fout, PA, PB)
    rng = np.random.default_rng(953)
    ii = np.concatenate([rng.integers(0, case.M, 4096), [0, 0, case.M - 1, case.M - 1]])
    jj = np.concatenate([rng.integers(0, case.N, 4096), [0, case.N - 1, 0, case.N - 1]])
    An, Bn = A.numpy(), B.numpy()
    ref, l1 = orc.matmul_acc_mx_at(An, case.fa, case.ta, Bn, case.fb, case.tb, PA.numpy(),
                                   PB.numpy(), ii, jj)
    _compare_acc(acc[ii, jj], ref, l1, case.K)
    check_p1(codes, e_out, amax, acc, case.K, case.a_scale_log2, case.b_scale_log2, case.fout)


@pytest.mark.parametrize("fout", [sc.E4M3, sc.E5M2])
def test_subnormal_accumulators_single_shift(fout):
    """Block factors of 2^-140 make every product, and so the accumulators,
    fp32 subnormals: P1 checks that the statistic and every code come from
    the GPU's accumulator through one power-of-two shift (reading R30), the
    case the plain FP8 path never reaches (its accumulators are >= 2^-32)."""
    M, N, K = 64, 80, 256
    say(f"case mx subnormal accumulators fout={fout}")
    A = _codes((M, K), sc.E4M3, 921)
    B = _codes((K, N), sc.E4M3, 922)
    ld = orc.mx_block_scale_ld(K)
    PA = torch.full((M, ld), 127 - 70, dtype=torch.uint8)
    PB = torch.full((N, ld), 127 - 70, dtype=torch.uint8)
    codes, e_out, amax, acc = _mx_run(A, 0, False, 60, B, 0, False, 60, fout, PA, PB)
    nz = acc[acc != 0]
    record("mx_subnormal", fout=FMT[fout], nonzero=int(nz.size),
           subnormal=int(np.count_nonzero(np.abs(nz) < 2.0 ** -126)), e_out=e_out)
    say(f"  nonzero acc {nz.size}, subnormal {np.count_nonzero(np.abs(nz) < 2.0 ** -126)}")
    assert nz.size > 0 and np.all(np.abs(nz) < 2.0 ** -126)
    check_p1(codes, e_out, amax, acc, K, 60, 60, fout)
    # P2 against the oracle's block-scaled sum (exact in fp64, one rounding)
    ref = orc.matmul_acc_mx(A.numpy(), 0, False, B.numpy(), 0, False, PA.numpy(), PB.numpy())
    l1 = orc.matmul_acc_mx(A.numpy() & 0x7F, 0, False, B.numpy() & 0x7F, 0, False,
                           PA.numpy(), PB.numpy())
    err = np.abs(acc.astype(np.float64) - ref.astype(np.float64))
    record("mx_subnormal_p2", fout=FMT[fout], max_err=float(err.max()),
           max_l1=float(l1.max()), exact=int(np.count_nonzero(err == 0)), n=int(err.size))
    say(f"  P2 max |acc - ref| {err.max():.3g} (l1 max {l1.max():.3g}), exact {np.count_nonzero(err == 0)}")


@pytest.mark.parametrize("mode", list(MODES))
@pytest.mark.parametrize("fout", [sc.E4M3, sc.E5M2, sc.F16])
def test_interior_path_equals_the_checked_path(mode, fout):
    """Block-scaled calls without an exported accumulator (interior wave
    tiles cast or stored without per-element checks, the single pass where
    it runs) give the codes, scale and statistic of the same call with the
    export, which P1 checks."""
    M, N, K = 512, 384, 512
    say(f"case mx interior {mode} fout={fout}")
    A = _codes((M, K), 0, 960)
    B = _codes((K, N), 1, 961)
    PA = wl.mx_block_scales(M, K, 962)
    PB = wl.mx_block_scales(N, K, 963)
    fast = _mx_run(A, 0, False, -1, B, 1, False, 2, fout, PA, PB, MODES[mode], amax_in=3.0,
                   want_acc=False)
    run = _mx_run(A, 0, False, -1, B, 1, False, 2, fout, PA, PB, MODES[mode], amax_in=3.0)
    assert np.array_equal(fast[0], run[0]), f"{np.count_nonzero(fast[0] != run[0])} codes differ"
    assert fast[1] == run[1] and np.float32(fast[2]) == np.float32(run[2])
    _check(run, A, 0, False, -1, B, 1, False, 2, fout, PA, PB, MODES[mode], amax_in=3.0)
