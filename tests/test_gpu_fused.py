"""GPU parity of scalify_matmul with the fused scaled add (Algorithm 3 rule)
and activation (Appendix C.1) in its epilogue, through the C ABI, against
the CPU oracle.

For each call the kernel exports its accumulator (acc_out) and the pre-cast
value w (pre_out). Checks:
  F1  w equals the oracle's fused pre-cast value computed from the GPU's own
      accumulator: bit for bit for the add and relu (exact arithmetic, one
      rounding of the sum); for gelu and silu, whose gate the kernel
      evaluates in fp32, within (16 + 4|t|) ulp of the oracle's fp64 value
      (t the sigmoid argument) plus |w_0| 2^-125 where the gate flushes;
  F2  codes, output scale and statistic equal the oracle's rescale and cast
      of the GPU's own w (exact);
  P2  the accumulator against the oracle's (as for the plain matmul).
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
ACTS = {"none": sc.ACT_NONE, "relu": sc.ACT_RELU, "gelu": sc.ACT_GELU_TANH, "silu": sc.ACT_SILU}
FMT_NAMES = {sc.E4M3: "e4m3", sc.E5M2: "e5m2", sc.F16: "f16"}


def _codes(shape, fmt, seed, heavy=False):
    return wl.fp8_normal(shape, fmt, seed, "cpu", 10.0 if heavy else None)


def _residual_codes(M, N, fmt, seed, rows=None, spread=None):
    """Residual code matrix [rows or M, N] (numpy; uint16 for F16)."""
    g = torch.Generator().manual_seed(seed)
    x = torch.randn((rows or M, N), generator=g, dtype=torch.float32)
    if spread is not None:
        x = x * torch.exp2(torch.randint(-spread, spread + 1, x.shape, generator=g).float())
    return orc.cast(fmt, x.numpy())


def _residual_device(codes, fmt, M):
    """Device ScaledArray data for a residual: padded rows (ld a multiple of
    16 elements), a [1, N] row expanded to [M, N] (stride 0) for a bias."""
    R, N = codes.shape
    if fmt == sc.F16:
        st = torch.full((R, max(16, (N + 15) // 16 * 16)), 0x7E00, dtype=torch.int16, device=DEV)
        st[:, :N] = torch.from_numpy(codes.view(np.int16)).to(DEV)
        d = st[:, :N]
    else:
        d = stored_with_padding(torch.from_numpy(codes), DEV)
    if R == 1 and M != 1:
        d = d.expand(M, N)
    return d


def _run(A, fa, ta, sa, B, fb, tb, sb, fout, *, res=None, act=sc.ACT_NONE, mode=sc.RESCALE_AMAX,
         target=0, sat=True, amax_in=0.0, inplace=False, want_pre=True, ch_a=None, ch_b=None):
    """One fused scalify_matmul call. res = (codes, fmt, scale_log2) or None;
    ch_a / ch_b: numpy channel scales ([M] / [N] powers of two) or None.
    Returns codes, e_out, amax, acc, pre (w), K."""
    a = sc.ScaledArray(stored_with_padding(A, DEV), fa, sc.scale_tensor(sa, DEV), ta)
    b = sc.ScaledArray(stored_with_padding(B, DEV), fb, sc.scale_tensor(sb, DEV), tb)
    M, K = a.shape
    N = b.shape[1]
    residual = None
    if res is not None:
        rcodes, rfmt, rq = res
        residual = sc.ScaledArray(_residual_device(rcodes, rfmt, M), rfmt, sc.scale_tensor(rq, DEV))
    if inplace:
        assert res is not None and res[1] == fout and res[0].shape[0] == M
        out = sc.ScaledArray(residual.data, fout, torch.empty(1, dtype=torch.float32, device=DEV))
    else:
        out = sc.empty_scaled(M, N, fout, DEV)
    acc = torch.empty((M, N), dtype=torch.float32, device=DEV)
    pre = torch.empty((M, N), dtype=torch.float32, device=DEV) if want_pre else None
    stat_in = torch.tensor([amax_in], dtype=torch.float32, device=DEV)
    stat_out = torch.empty(1, dtype=torch.float32, device=DEV)
    sc.scalify_matmul(a, b, out, rescale=mode, target_log2=target, saturate=sat, acc_out=acc,
                      amax_out=stat_out, amax_in=stat_in if mode == sc.RESCALE_DELAYED else None,
                      residual=residual, activation=act, pre_out=pre,
                      a_channel_scale=_dev_f32(ch_a), b_channel_scale=_dev_f32(ch_b))
    torch.cuda.synchronize()
    codes = out.data.cpu().numpy()
    if fout == sc.F16:
        codes = codes.view(np.uint16)
    s = float(out.scale.item())
    e_out = int(math.frexp(s)[1] - 1)
    assert s == 2.0 ** e_out
    return (codes.copy(), e_out, float(stat_out.item()), acc.cpu().numpy(),
            pre.cpu().numpy() if want_pre else None, K)


def _dev_f32(x):
    return None if x is None else torch.from_numpy(np.asarray(x, dtype=np.float32)).to(DEV)


def _oracle_res(res):
    if res is None:
        return None
    codes, fmt, q = res
    return codes, fmt, 2.0 ** q


def _gate_arg(act, x):
    """Argument of the sigmoid the kernel evaluates (x for silu, 2u for the
    tanh form of gelu), for the fp32 error bound only."""
    with np.errstate(over="ignore", invalid="ignore"):
        if act == sc.ACT_GELU_TANH:
            return 2.0 * math.sqrt(2.0 / math.pi) * (x + 0.044715 * x ** 3)
        return x


def check_fused(run, sa, sb, fout, res, act, mode, target=0, sat=True, amax_in=0.0, ch_a=None,
                ch_b=None):
    """F1 and F2 for one call's outputs; returns the number of elements of w
    that differ from the oracle's value (gelu / silu only)."""
    codes, e_out, amax, acc, pre, K = run
    ores = _oracle_res(res)
    w_ref, y64, e_w, e_cc = orc.fused_pre(acc, 2.0 ** sa, 2.0 ** sb, K, ores, act, ch_a, ch_b)
    # F1
    nan_g, nan_r = np.isnan(pre), np.isnan(y64)
    assert np.array_equal(nan_g, nan_r), "F1: NaN pattern of w differs"
    if act in (sc.ACT_NONE, sc.ACT_RELU):
        assert np.array_equal(pre.view(np.uint32)[~nan_g], w_ref.view(np.uint32)[~nan_g]), \
            f"F1: w differs at {np.flatnonzero((pre != w_ref) & ~nan_g)[:5]}"
        n_diff = 0
    else:
        w0, _, _, _ = orc.fused_pre(acc, 2.0 ** sa, 2.0 ** sb, K, ores, sc.ACT_NONE, ch_a, ch_b)
        fin = ~nan_r
        x = w0.astype(np.float64)[fin] * 2.0 ** e_w
        t = np.abs(_gate_arg(act, x))
        t = np.where(np.isfinite(t), t, 0.0)     # the gate is exactly 0 or 1 there
        tol = np.abs(y64[fin]) * (16.0 + 4.0 * t) * 2.0 ** -24 + np.abs(w0[fin]) * 2.0 ** -125
        inf = np.isinf(y64[fin])
        assert np.array_equal(pre[fin][inf], y64[fin][inf]), "F1: Inf of w differs"
        err = np.abs(pre[fin][~inf].astype(np.float64) - y64[fin][~inf])
        assert np.all(err <= tol[~inf]), \
            f"F1: worst err/tol {float((err / np.maximum(tol[~inf], 1e-300)).max())}"
        n_diff = int((pre[fin] != w_ref[fin]).sum())
    # F2
    ref_codes, ref_e, ref_amax = orc.finish_pre(pre, e_w, e_cc, mode, target, amax_in, sat, fout)
    assert e_out == ref_e, (e_out, ref_e)
    assert np.float32(amax) == np.float32(ref_amax), (amax, ref_amax)
    bad = np.flatnonzero(codes.ravel() != ref_codes.ravel())
    assert bad.size == 0, f"F2: {bad.size} mismatches, first {bad[:5]} gpu " \
        f"{codes.ravel()[bad[:5]]} ref {ref_codes.ravel()[bad[:5]]} w {pre.ravel()[bad[:5]]}"
    return n_diff


# (activation, residual format or None, broadcast row)
COMBOS = [("relu", None, False), ("gelu", None, False), ("silu", None, False),
          ("none", sc.E4M3, False), ("none", sc.E5M2, False), ("none", sc.F16, False),
          ("none", sc.E4M3, True), ("relu", sc.E5M2, False), ("gelu", sc.E4M3, True),
          ("silu", sc.F16, False)]
SHAPES = [(1, 1, 1), (17, 33, 65), (257, 513, 129), (300, 200, 1000)]
MODES = {"amax": sc.RESCALE_AMAX, "none": sc.RESCALE_NONE, "delayed": sc.RESCALE_DELAYED}
LAYOUTS = list(itertools.product((False, True), repeat=2))


@pytest.mark.parametrize("mode", list(MODES))
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("combo", COMBOS,
                         ids=lambda c: f"{c[0]}-{FMT_NAMES[c[1]] if c[1] is not None else 'nores'}"
                                       f"{'-bias' if c[2] else ''}")
def test_fused_parity(combo, shape, mode):
    act_name, rfmt, bias = combo
    act = ACTS[act_name]
    M, N, K = shape
    i = COMBOS.index(combo) + 3 * SHAPES.index(shape)
    ta, tb = LAYOUTS[i % 4]
    fa, fb = [(0, 0), (1, 0), (0, 1), (1, 1)][(i // 2) % 4]
    fout = [sc.E4M3, sc.E5M2, sc.F16][i % 3]
    sa, sb, q = -2, 1, [3, -4, 0, 7][i % 4]
    say(f"case fused {act_name} res={rfmt} bias={bias} {shape} {mode} ta={ta} tb={tb} "
        f"fmts={fa},{fb}->{fout} q={q}")
    A = _codes((K, M) if ta else (M, K), fa, 500 + M + i, heavy=fa == sc.E5M2)
    B = _codes((N, K) if tb else (K, N), fb, 600 + N + i, heavy=fb == sc.E5M2)
    res = None
    if rfmt is not None:
        res = (_residual_codes(M, N, rfmt, 700 + i, rows=1 if bias else None, spread=4), rfmt, q)
    amax_in = 5.0 if mode == "delayed" else 0.0
    run = _run(A, fa, ta, sa, B, fb, tb, sb, fout, res=res, act=act, mode=MODES[mode],
               amax_in=amax_in)
    n = check_fused(run, sa, sb, fout, res, act, MODES[mode], amax_in=amax_in)
    if shape == (257, 513, 129) and mode == "amax":
        check_p2_full(run[3], A, fa, ta, B, fb, tb)
    say(f"  ok, {n} gate values off the oracle's fp32 rounding")


@pytest.mark.parametrize("mode", [sc.RESCALE_AMAX, sc.RESCALE_NONE, sc.RESCALE_DELAYED])
@pytest.mark.parametrize("fout", [sc.E4M3, sc.E5M2, sc.F16])
def test_fused_kernel_with_nothing_fused_equals_the_plain_kernel(mode, fout):
    """pre_out alone selects the fused kernels (fp32 intermediate): the codes,
    scale and statistic must be the plain kernels' bit for bit, and w = acc."""
    say(f"case fused-identity mode={mode} fout={fout}")
    A = _codes((300, 700), sc.E4M3, 31)
    B = _codes((700, 260), sc.E4M3, 32)
    kw = dict(mode=mode, amax_in=2.0 ** -3)
    fused = _run(A, 0, False, 2, B, 0, False, -5, fout, **kw)
    plain = _run(A, 0, False, 2, B, 0, False, -5, fout, want_pre=False, **kw)
    assert np.array_equal(fused[0], plain[0]) and fused[1] == plain[1] and fused[2] == plain[2]
    assert np.array_equal(fused[4].view(np.uint32), plain[3].view(np.uint32))


@pytest.mark.parametrize("mode", [sc.RESCALE_AMAX, sc.RESCALE_DELAYED])
@pytest.mark.parametrize("fout", [sc.E4M3, sc.F16])
def test_fused_residual_in_place(mode, fout):
    """out and the residual are the very same matrix (x <- x + f(x) W style):
    same codes and scale as writing to a separate output."""
    say(f"case fused in-place mode={mode} fout={fout}")
    M, N, K = 260, 300, 512
    A = _codes((M, K), sc.E4M3, 41)
    B = _codes((K, N), sc.E4M3, 42)
    res = (_residual_codes(M, N, fout, 43), fout, 2)
    sep = _run(A, 0, False, 0, B, 0, False, 0, fout, res=res, act=sc.ACT_GELU_TANH, mode=mode,
               amax_in=3.0)
    inp = _run(A, 0, False, 0, B, 0, False, 0, fout, res=res, act=sc.ACT_GELU_TANH, mode=mode,
               amax_in=3.0, inplace=True)
    assert np.array_equal(sep[0], inp[0]) and sep[1] == inp[1] and sep[2] == inp[2]
    check_fused(inp, 0, 0, fout, res, sc.ACT_GELU_TANH, mode, amax_in=3.0)


@pytest.mark.parametrize("mode", [sc.RESCALE_AMAX, sc.RESCALE_DELAYED])
def test_fused_specials(mode):
    """NaN / Inf residual codes (E5M2), NaN accumulators, gates at a scaled
    value beyond the fp32 range (x * 2^e_w overflows) and near zero."""
    say(f"case fused specials mode={mode}")
    M, N, K = 64, 96, 256
    A = _codes((M, K), sc.E5M2, 51, heavy=True).numpy().copy()
    B = _codes((K, N), sc.E4M3, 52).numpy().copy()
    A[5, 9] = 0x7F                                     # NaN row
    A_t, B_t = torch.from_numpy(A), torch.from_numpy(B)
    r = _residual_codes(M, N, sc.E5M2, 53)
    r[0, :8] = [0x7C, 0xFC, 0x7D, 0xFE, 0x00, 0x80, 0x7B, 0xFB]  # +-Inf, NaNs, +-0, +-max
    res = (r, sc.E5M2, -3)
    for act in (sc.ACT_RELU, sc.ACT_GELU_TANH, sc.ACT_SILU):
        for sa, sb in [(0, 0), (100, 27), (-60, -60)]:
            run = _run(A_t, sc.E5M2, False, sa, B_t, sc.E4M3, False, sb, sc.E5M2, res=res, act=act,
                       mode=mode, amax_in=1.0)
            check_fused(run, sa, sb, sc.E5M2, res, act, mode, amax_in=1.0)
            run = _run(A_t, sc.E5M2, False, sa, B_t, sc.E4M3, False, sb, sc.E4M3, act=act,
                       mode=mode, amax_in=1.0)
            check_fused(run, sa, sb, sc.E4M3, None, act, mode, amax_in=1.0)


def test_fused_gate_tails_with_a_tiny_output():
    """silu far in its negative tail (x * 2^e_w from -40 to -130): gates from
    about 2^-58 down to fp32 underflow, an output whose amax is tiny, and a
    rescale that scales w up by more than 2^90."""
    say("case fused gate tails")
    M, N, K = 16, 64, 1
    A = orc.cast(sc.E4M3, np.ones((M, K), dtype=np.float32))
    xs = -np.linspace(40.0, 130.0, N).astype(np.float32)
    B = orc.cast(sc.E4M3, xs[None, :] / 16.0)
    A_t, B_t = torch.from_numpy(A), torch.from_numpy(B)
    for mode in (sc.RESCALE_AMAX, sc.RESCALE_DELAYED):
        for fout in (sc.E4M3, sc.E5M2, sc.F16):
            run = _run(A_t, 0, False, 2, B_t, 0, False, 2, fout, act=sc.ACT_SILU, mode=mode,
                       amax_in=2.0 ** -80)
            check_fused(run, 2, 2, fout, None, sc.ACT_SILU, mode, amax_in=2.0 ** -80)


@pytest.mark.parametrize("fout", [sc.E4M3, sc.E5M2, sc.F16])
def test_fused_subnormal_pre_cast_values_cast_exactly(fout):
    """K = 0 and a residual whose scale is 2^-130 of the product's: w =
    r * 2^-130 is an fp32 subnormal, the statistic is itself subnormal and the
    rescale scales w back up by 2^127 (clamped output scale), so the casts
    of subnormal fp32 values decide every code."""
    say(f"case fused subnormal w fout={fout}")
    M, N = 24, 80
    rc = _residual_codes(M, N, sc.E4M3, 85, spread=3)
    res = (rc, sc.E4M3, -30)
    A = torch.zeros((M, 0), dtype=torch.uint8)
    B = torch.zeros((0, N), dtype=torch.uint8)
    for mode, amax_in in [(sc.RESCALE_AMAX, 0.0), (sc.RESCALE_NONE, 0.0),
                          (sc.RESCALE_DELAYED, 2.0 ** -127)]:
        run = _run(A, 0, False, 50, B, 0, False, 50, fout, res=res, mode=mode, amax_in=amax_in)
        pre = run[4]
        assert np.any((pre != 0) & (np.abs(pre) < 2.0 ** -126))
        check_fused(run, 50, 50, fout, res, sc.ACT_NONE, mode, amax_in=amax_in)


@pytest.mark.parametrize("fout", [sc.E4M3, sc.E5M2, sc.F16])
@pytest.mark.parametrize("mode", [sc.RESCALE_AMAX, sc.RESCALE_DELAYED])
def test_fused_integer_grid_end_to_end_exact(fout, mode):
    """Integer-valued operands and residual (exact accumulators and sums):
    the whole relu(A B + R) path equals the oracle's end to end, from the
    oracle's own accumulator, with no exemption."""
    say(f"case fused grid fout={fout} mode={mode}")
    M, N, K = 300, 260, 1000
    A = wl.int_grid((M, K), sc.E4M3, 71)
    B = wl.int_grid((K, N), sc.E4M3, 72)
    rc = orc.cast(sc.E4M3, np.random.default_rng(73).integers(-8, 9, (M, N)).astype(np.float32))
    res = (rc, sc.E4M3, 9)
    run = _run(A, 0, False, 0, B, 0, False, 0, fout, res=res, act=sc.ACT_RELU, mode=mode,
               amax_in=2.0 ** 6)
    acc_ref = orc.matmul_acc(A.numpy(), 0, False, B.numpy(), 0, False)
    assert np.array_equal(run[3], acc_ref)
    codes, e_out, amax, _, _ = orc.matmul_epilogue_fused(acc_ref, 1.0, 1.0, K, (rc, sc.E4M3, 2.0 ** 9),
                                                         sc.ACT_RELU, mode, 0, 2.0 ** 6, True, fout)
    assert np.array_equal(run[0], codes) and run[1] == e_out and run[2] == amax


def test_fused_empty_and_k_zero():
    """K = 0: the output is the residual alone (scaled add with a zero
    product); M = 0 or N = 0: nothing to do."""
    say("case fused empty")
    M, N = 33, 48
    rc = _residual_codes(M, N, sc.E4M3, 81)
    res = (rc, sc.E4M3, 4)
    for mode in (sc.RESCALE_AMAX, sc.RESCALE_NONE):
        run = _run(torch.zeros((M, 0), dtype=torch.uint8), 0, False, 0,
                   torch.zeros((0, N), dtype=torch.uint8), 0, False, 0, sc.E4M3, res=res,
                   act=sc.ACT_RELU, mode=mode)
        check_fused(run, 0, 0, sc.E4M3, res, sc.ACT_RELU, mode)
        assert np.all(run[3] == 0)
    for M_, N_ in [(0, 16), (16, 0)]:
        run = _run(torch.zeros((M_, 32), dtype=torch.uint8), 0, False, 0,
                   torch.zeros((32, N_), dtype=torch.uint8), 0, False, 0, sc.E4M3,
                   res=(np.zeros((M_, N_), dtype=np.uint8), sc.E4M3, 0), act=sc.ACT_SILU)
        assert run[0].size == 0


@pytest.mark.parametrize("size", [8192])
def test_fused_square_full_size(size):
    """The square workload at full size with a residual add and gelu, in the
    launch configuration the benchmark times: F1 and F2 on every element
    (from the GPU's accumulator), P2 of the accumulator on a sample."""
    from tests.helpers import check_p2_sampled
    case = wl.config_4(size, wl.E4M3)[0]
    say(f"case fused {case.name} gelu + residual")
    A, B = case.make_a("cpu"), case.make_b("cpu")
    res = (_residual_codes(size, size, sc.E4M3, 91), sc.E4M3, case.a_scale_log2 + 3)
    run = _run(A, case.fa, False, case.a_scale_log2, B, case.fb, False, case.b_scale_log2,
               case.fout, res=res, act=sc.ACT_GELU_TANH)
    n = check_fused(run, case.a_scale_log2, case.b_scale_log2, case.fout, res, sc.ACT_GELU_TANH,
                    sc.RESCALE_AMAX)
    check_p2_sampled(run[3], A, case.fa, False, B, case.fb, False, n_samples=4096)
    say(f"  ok: {n} of {size * size} gate values off the oracle's fp32 rounding")
