"""GPU parity of scalify_rescale / scalify_cast / scalify_set_scaling (through
the C ABI) against the CPU oracle: codes and output scales bit-exact."""
import numpy as np
import pytest
import torch

from oracle import oracle as orc
from paper_2407_17353_amd import binding as sc
from tests.helpers import say

pytestmark = pytest.mark.gpu

DEV = "cuda"
NP_STORE = {sc.E4M3: np.uint8, sc.E5M2: np.uint8, sc.F16: np.uint16, sc.F32: np.float32}


def _to_device(x_np, fmt, rows, cols):
    if fmt == sc.F16:
        t = torch.from_numpy(x_np.view(np.int16).reshape(rows, cols))
    else:
        t = torch.from_numpy(x_np.reshape(rows, cols))
    return t.to(DEV)


def _from_device(t, fmt):
    a = t.cpu().numpy()
    return a.view(np.uint16) if fmt == sc.F16 else a


def _inputs(fmt, n, seed):
    """Random data with the specials mixed in."""
    rng = np.random.default_rng(seed)
    if fmt == sc.F32:
        x = (rng.standard_normal(n) * np.exp2(rng.uniform(-30, 30, n))).astype(np.float32)
        x[:8] = [0.0, -0.0, np.inf, -np.inf, np.nan, 1e-45, -3e38, 65520.0]
        return x
    if fmt == sc.F16:
        x = rng.integers(0, 65536, n).astype(np.uint16)
        return x
    return rng.integers(0, 256, n).astype(np.uint8)


def _out_empty(rows, cols, fmt):
    return sc.ScaledArray(torch.empty((rows, cols), dtype=sc.STORAGE_DTYPE[fmt], device=DEV), fmt,
                          torch.empty(1, dtype=torch.float32, device=DEV))


@pytest.mark.parametrize("in_fmt", [sc.E4M3, sc.E5M2, sc.F16, sc.F32])
@pytest.mark.parametrize("out_fmt", [sc.E4M3, sc.E5M2, sc.F16])
@pytest.mark.parametrize("mode", [sc.RESCALE_AMAX, sc.RESCALE_NONE])
def test_rescale_matches_oracle(in_fmt, out_fmt, mode):
    rows, cols = 37, 1777  # n = 65749: many 16-element chunks plus a ragged tail
    n = rows * cols
    say(f"case rescale in={in_fmt} out={out_fmt} mode={mode}")
    x = _inputs(in_fmt, n, 1000 + 10 * in_fmt + out_fmt)
    # avoid NaN-only / Inf-dominated amax in most cases: drop Inf codes for AMAX
    xin = sc.ScaledArray(_to_device(x, in_fmt, rows, cols), in_fmt, sc.scale_tensor(-5, DEV))
    out = _out_empty(rows, cols, out_fmt)
    for sat in (True, False):
        sc.scalify_rescale(xin, out, mode=mode, target_log2=1, saturate=sat)
        torch.cuda.synchronize()
        ref, e_ref, _ = orc.rescale(x, in_fmt, 2.0 ** -5, mode, 1, sat, out_fmt)
        got = _from_device(out.data, out_fmt).ravel()
        assert out.scale.item() == 2.0 ** e_ref
        bad = np.flatnonzero(got != ref)
        assert bad.size == 0, (bad[:5], got[bad[:5]], ref[bad[:5]])


@pytest.mark.parametrize("in_fmt", [sc.F32, sc.F16])
@pytest.mark.parametrize("out_fmt", [sc.E4M3, sc.E5M2])
def test_rescale_finite_inputs(in_fmt, out_fmt):
    """Finite data only, so the amax is a real statistic (no Inf)."""
    rows, cols = 512, 1031
    n = rows * cols
    rng = np.random.default_rng(77)
    v = (rng.standard_normal(n) * 3e-3).astype(np.float32)
    x = v if in_fmt == sc.F32 else v.astype(np.float16).view(np.uint16)
    say(f"case finite rescale in={in_fmt} out={out_fmt}")
    xin = sc.ScaledArray(_to_device(x, in_fmt, rows, cols), in_fmt, sc.scale_tensor(7, DEV))
    out = _out_empty(rows, cols, out_fmt)
    sc.scalify_rescale(xin, out)
    torch.cuda.synchronize()
    ref, e_ref, amax = orc.rescale(x, in_fmt, 2.0 ** 7, orc.RESCALE_AMAX, 0, True, out_fmt)
    assert out.scale.item() == 2.0 ** e_ref
    assert np.array_equal(_from_device(out.data, out_fmt).ravel(), ref)
    dec = orc.decode(out_fmt, ref)
    assert 1.0 <= np.abs(dec).max() < 2.0 + 1e-9


def test_rescale_in_place():
    rows, cols = 64, 1024
    x = _inputs(sc.E4M3, rows * cols, 5)
    x[x == 0x7F] = 0
    x[x == 0xFF] = 0
    t = _to_device(x, sc.E4M3, rows, cols)
    s = sc.scale_tensor(3, DEV)
    arr = sc.ScaledArray(t, sc.E4M3, s)
    say("case in-place rescale")
    sc.scalify_rescale(arr, arr, target_log2=4)
    torch.cuda.synchronize()
    ref, e_ref, _ = orc.rescale(x, sc.E4M3, 8.0, orc.RESCALE_AMAX, 4, True, sc.E4M3)
    assert s.item() == 2.0 ** e_ref
    assert np.array_equal(t.cpu().numpy().ravel(), ref)


def _structured_f32(exp_lo, exp_hi, top_bits, lows):
    low_n = 23 - top_bits
    exps = np.arange(exp_lo, exp_hi + 1, dtype=np.uint32)
    tops = np.arange(1 << top_bits, dtype=np.uint32)
    lw = np.array(lows, dtype=np.uint32) & ((1 << low_n) - 1)
    e, t, l = np.meshgrid(exps, tops, lw, indexing="ij")
    bits = ((e << 23) | (t << low_n) | l).ravel()
    bits = np.concatenate([bits, bits | np.uint32(0x80000000),
                           np.array([0, 0x80000000, 0x7F800000, 0xFF800000, 0x7FC00000, 0x7F800001,
                                     0xFFC00000, 1, 0x807FFFFF], dtype=np.uint32)])
    return bits.view(np.float32)


@pytest.mark.parametrize("out_fmt", [sc.E4M3, sc.E5M2, sc.F16])
def test_cast_f32_structured_exhaustive_rounding(out_fmt):
    """Every exponent from 2^-40 to 2^20, every value of the top mantissa
    bits, and the low-bit patterns that decide ties and sticky bits; both
    saturation modes."""
    top = 11 if out_fmt == sc.F16 else 9
    low_n = 23 - top
    lows = [0, 1, 2, (1 << (low_n - 1)) - 1, 1 << (low_n - 1), (1 << (low_n - 1)) + 1,
            (1 << low_n) - 2, (1 << low_n) - 1]
    x = _structured_f32(127 - 40, 127 + 20, top, lows)
    n = x.size - x.size % 16 + 16
    x = np.concatenate([x, np.zeros(n - x.size, np.float32)])
    rows = 16
    cols = n // rows
    say(f"case structured cast out={out_fmt} n={n}")
    xin = sc.ScaledArray(_to_device(x, sc.F32, rows, cols), sc.F32, sc.scale_tensor(-9, DEV))
    out = _out_empty(rows, cols, out_fmt)
    for sat in (True, False):
        sc.scalify_cast(xin, out, saturate=sat)
        torch.cuda.synchronize()
        got = _from_device(out.data, out_fmt).ravel()
        ref = orc.cast(out_fmt, x, saturate=sat)
        bad = np.flatnonzero(got != ref)
        assert bad.size == 0, (x[bad[:5]], got[bad[:5]], ref[bad[:5]])
        assert out.scale.item() == 2.0 ** -9


@pytest.mark.parametrize("in_fmt,out_fmt", [(sc.E4M3, sc.F16), (sc.E5M2, sc.F16), (sc.F16, sc.E4M3),
                                            (sc.E5M2, sc.E4M3), (sc.E4M3, sc.E5M2)])
def test_cast_all_codes(in_fmt, out_fmt):
    n = 65536 if in_fmt == sc.F16 else 256
    x = np.arange(n).astype(NP_STORE[in_fmt])
    say(f"case all-code cast {in_fmt}->{out_fmt}")
    xin = sc.ScaledArray(_to_device(x, in_fmt, 16, n // 16), in_fmt, None)
    out = _out_empty(16, n // 16, out_fmt)
    sc.scalify_cast(xin, out)
    torch.cuda.synchronize()
    assert out.scale.item() == 1.0
    assert np.array_equal(_from_device(out.data, out_fmt).ravel(), orc.cast_data(x, in_fmt, out_fmt))


@pytest.mark.parametrize("e_new", [-127, -20, -3, 0, 6, 40, 127])
def test_set_scaling(e_new):
    rows, cols = 8, 4000
    x = _inputs(sc.F32, rows * cols, 9)
    say(f"case set_scaling e_new={e_new}")
    xin = sc.ScaledArray(_to_device(x, sc.F32, rows, cols), sc.F32, sc.scale_tensor(2, DEV))
    for out_fmt in (sc.E4M3, sc.E5M2, sc.F16):
        out = _out_empty(rows, cols, out_fmt)
        sc.scalify_set_scaling(xin, out, e_new)
        torch.cuda.synchronize()
        assert out.scale.item() == 2.0 ** e_new
        ref = orc.set_scaling(x, sc.F32, 4.0, e_new, True, out_fmt)
        assert np.array_equal(_from_device(out.data, out_fmt).ravel(), ref)


def test_rescale_large_bench_size():
    """fp32 [8192, 8192] -> E4M3, the standalone rescale/cast at full size."""
    rows = cols = 8192
    g = torch.Generator(device=DEV)
    g.manual_seed(3)
    x = torch.randn((rows, cols), generator=g, device=DEV) * 1e-2
    say("case large rescale 8192^2")
    xin = sc.ScaledArray(x, sc.F32, sc.scale_tensor(0, DEV))
    out = _out_empty(rows, cols, sc.E4M3)
    sc.scalify_rescale(xin, out)
    torch.cuda.synchronize()
    xn = x.cpu().numpy().ravel()
    ref, e_ref, _ = orc.rescale(xn, sc.F32, 1.0, orc.RESCALE_AMAX, 0, True, sc.E4M3)
    assert out.scale.item() == 2.0 ** e_ref
    assert np.array_equal(out.data.cpu().numpy().ravel(), ref)
