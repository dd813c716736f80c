"""scalify_matmul_noalloc (the allocation-free entry point, workspace in the
library's static device array) against scalify_matmul with a caller-owned
workspace, through the C ABI: codes, output scale and statistic bit for bit
on consecutive calls whose sizes shrink (the array keeps the previous call's
contents, so every value the kernels need cleared must be cleared by the
call itself), in the dynamic, static and delayed modes, and the refusal of
calls whose workspace exceeds the array."""
import math

import numpy as np
import pytest
import torch

from paper_2407_17353_amd import binding as sc
from paper_2407_17353_amd import workloads as wl
from tests.helpers import say, stored_with_padding

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _operands(M, N, K, fa, fb, seed):
    # rows padded to 16 bytes (the matmul's alignment rule), padding NaN
    A = stored_with_padding(wl.fp8_normal((M, K), fa, seed, DEV), DEV)
    B = stored_with_padding(wl.fp8_normal((K, N), fb, seed + 1, DEV), DEV)
    a = sc.ScaledArray(A, fa, sc.scale_tensor(-2, DEV))
    b = sc.ScaledArray(B, fb, sc.scale_tensor(3, DEV))
    return a, b


def _call(fn, a, b, M, N, fout, mode, **kw):
    out = sc.empty_scaled(M, N, fout, DEV)
    out.data.fill_(0x33)
    stat = torch.full((1,), 5.0, dtype=torch.float32, device=DEV)
    amax = torch.full((1,), -1.0, dtype=torch.float32, device=DEV)
    if mode == sc.RESCALE_DELAYED:
        kw["amax_in"] = stat
    fn(a, b, out, rescale=mode, amax_out=amax, **kw)
    torch.cuda.synchronize()
    codes = out.data.cpu().numpy()
    if fout == sc.F16:
        codes = codes.view(np.uint16)
    return codes.copy(), float(out.scale.item()), float(amax.item())


# (M, N, K, fa, fb, fout, mode): each list is run in order, sizes shrinking
SEQUENCES = {
    "amax": [(2048, 4096, 1024, 0, 0, sc.E4M3, sc.RESCALE_AMAX),
             (300, 520, 384, 1, 0, sc.E5M2, sc.RESCALE_AMAX)],
    "none_f16": [(1024, 2048, 640, 0, 1, sc.F16, sc.RESCALE_NONE),
                 (257, 129, 65, 0, 0, sc.F16, sc.RESCALE_NONE)],
    "delayed": [(8192, 8192, 512, 0, 0, sc.E4M3, sc.RESCALE_DELAYED),
                (1000, 777, 333, 1, 1, sc.E5M2, sc.RESCALE_DELAYED)],
}


@pytest.mark.parametrize("name", list(SEQUENCES))
def test_noalloc_matches_workspace_call_on_shrinking_calls(name):
    for i, (M, N, K, fa, fb, fout, mode) in enumerate(SEQUENCES[name]):
        say(f"case noalloc {name} call {i}: {M}x{N}x{K} fa={fa} fb={fb} fout={fout} mode={mode}")
        a, b = _operands(M, N, K, fa, fb, 1000 + 7 * i + M)
        ref = _call(sc.scalify_matmul, a, b, M, N, fout, mode)
        got = _call(sc.scalify_matmul_noalloc, a, b, M, N, fout, mode)
        assert got[1] == ref[1] and math.frexp(got[1])[0] == 0.5
        assert np.float32(got[2]) == np.float32(ref[2])
        bad = np.flatnonzero(got[0].ravel() != ref[0].ravel())
        assert bad.size == 0, f"{bad.size} codes differ, first {bad[:5]}"


def test_noalloc_refuses_a_workspace_beyond_its_array():
    """8192 x 8192 with the dynamic rescale needs a 128 MiB intermediate:
    refused with SCALIFY_ERR_WORKSPACE, the output left untouched."""
    say("case noalloc too large")
    M = N = 8192
    a, b = _operands(M, N, 128, 0, 0, 77)
    out = sc.empty_scaled(M, N, sc.E4M3, DEV)
    out.data.fill_(0x33)
    out.scale.fill_(7.0)
    with pytest.raises(sc.ScalifyError) as e:
        sc.scalify_matmul_noalloc(a, b, out)
    assert e.value.status == 6
    torch.cuda.synchronize()
    assert bool((out.data == 0x33).all()) and out.scale.item() == 7.0
