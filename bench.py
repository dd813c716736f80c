#!/usr/bin/env python3
"""Benchmark of the scaled-FP8 matmul with fused dynamic rescale and cast.

One step = one scalify_matmul call on the headline workload: M = N = K = 8192,
E4M3 x E4M3 -> E4M3 with the amax rescale (prologue + fused GEMM/amax +
epilogue cast), inputs already resident in HBM. Prints ONE JSON line with
the whole-call throughput (TFLOP/s), the roofline of the dominant kernel
(the fused GEMM, timed live with HIP events recorded by the library on its
stream) and the CPU oracle timed on a bounded sample of the same workload.
Before the W warm-up calls, the call runs back to back, untimed, until its
duration is steady (the chip's clock dips for the first calls of a process);
the line's `settle` object records that phase.

  python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-cpu-baseline]
  python bench.py --sweep      # also time every benchmark configuration
  python bench.py --copy-calibration   # also run a 256 MiB device copy (PMC scale)

`roofline.traffic` (HBM bytes per launch of the fused GEMM) comes from the
rocprofv3 FETCH_SIZE / WRITE_SIZE summary committed under profiles/, and is
reported only while the GEMM sources still hash to the value recorded there.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "scaled-FP8 GEMM TFLOP/s incl. rescale+cast; % of MI355X FP8 MFMA peak"
PEAK_FP8_TFLOPS = 5000.0      # MI355X dense FP8 MFMA, 256 CU x 2.4 GHz x 8192 FLOP/clk
PEAK_HBM_GBS = 8000.0
EVENT_EVERY = 4               # GEMM-bracketing events on every 4th timed call
FMT_NAME = {0: "e4m3", 1: "e5m2", 2: "f16"}
GEMM_SOURCES = ("paper_2407_17353_amd/csrc/gemm4_kernel.h", "paper_2407_17353_amd/csrc/gemm_kernel.h",
                "paper_2407_17353_amd/csrc/gemm_nn.hip", "paper_2407_17353_amd/csrc/ew_util.h",
                "paper_2407_17353_amd/csrc/codec.h", "paper_2407_17353_amd/csrc/kernels.h")
TRAFFIC_SUMMARY = "profiles/gemm_8192cube_e4m3_hbm_traffic.md"


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=100)
    p.add_argument("--warmup", type=int, default=100)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=12.0,
                   help="target CPU time of the oracle sample")
    p.add_argument("--sweep", action="store_true", help="also time every configuration")
    p.add_argument("--copy-calibration", action="store_true",
                   help="also run a plain 256 MiB device-to-device copy 5 times (the known-size "
                        "kernel that scales rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    return p.parse_args()


def gemm_source_hash():
    h = hashlib.sha256()
    for rel in GEMM_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic():
    """HBM bytes per launch of the 8192^3 GEMM from the committed rocprofv3
    summary, or None when it is missing or was taken on other GEMM sources."""
    path = os.path.join(ROOT, TRAFFIC_SUMMARY)
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_hash = re.search(r"gemm source hash: ([0-9a-f]{16})", text)
    m_bytes = re.search(r"HBM bytes per launch: ([0-9]+)", text)
    if not m_hash or not m_bytes or m_hash.group(1) != gemm_source_hash():
        return None
    return int(m_bytes.group(1))


def copy_calibration(dev, nbytes=256 << 20, reps=5):
    """A plain device copy of known size, for scaling the PMC byte counters."""
    import torch
    src = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


def settled(means, calls, min_calls=150, tol=0.01):
    """The settling rule: at least min_calls calls made, and the last two
    chunk means (ms) within tol of each other."""
    return calls >= min_calls and len(means) >= 2 and abs(means[-1] - means[-2]) <= tol * means[-2]


def settle_clock(call, stream, min_calls=150, max_calls=500, chunk=10, tol=0.01):
    """Run `call` back to back until its duration is steady: at least
    min_calls calls, then until two consecutive `chunk`-call means agree
    within `tol` (at most max_calls). In a fresh process the chip's clock
    first dips under the sustained FP8 matrix load (the first ~60 calls of
    the 8192^3 GEMM run up to 37 % slower at the same cycle count) and then
    settles; this runs before the warm-up calls, untimed, and its record
    (calls made, the first calls' and the slowest and last chunk's mean
    duration, every chunk's mean) goes into the bench line."""
    import torch
    means, first, n = [], [], 0
    while n < max_calls:
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(chunk + 1)]
        ev[0].record(stream)
        for i in range(chunk):
            call()
            ev[i + 1].record(stream)
        torch.cuda.synchronize()
        ts = [ev[i].elapsed_time(ev[i + 1]) for i in range(chunk)]
        first = first or ts
        means.append(sum(ts) / chunk)
        n += chunk
        if settled(means, n, min_calls, tol):
            break
    return {"calls": n, "first_calls_us": [round(t * 1e3, 1) for t in first[:5]],
            "slowest_10_call_mean_us": round(max(means) * 1e3, 1),
            "last_10_call_mean_us": round(means[-1] * 1e3, 1),
            "10_call_means_us": [round(m * 1e3) for m in means]}


def time_case(case, steps, warmup, dev, ws=None, mode=None, act=0, residual_seed=None,
              mx_seed=None, settle=False):
    """Time `steps` scalify_matmul calls of one GemmCase. Returns a dict with
    ms per call (event-timed over the whole timed region), the mean and the
    p10/p50/p90 duration of the fused GEMM kernel (events recorded by the
    library right before and after that launch, on every EVENT_EVERY-th call
    of the timed region), and,
    from a short pass after the timed region that also records an event
    after the epilogue, the mean epilogue-cast duration. Only the GEMM is
    bracketed in the timed region because every recorded event costs the
    stream a few microseconds. mode RESCALE_DELAYED keeps the statistic in
    one device word that every call reads and rewrites (model state).
    act / residual_seed: fuse that activation and, when residual_seed is
    given, the scaled add of a seeded E4M3 N(0,1) residual [M, N] (scale 2)
    into the GEMM epilogue. mx_seed: give A and B seeded MX block scales
    (E8M0 bytes per 32 k, exponents in [-8, 8]). settle: before the warm-up,
    run the call until the clock has settled (settle_clock; its record is
    returned under "settle")."""
    import torch
    from paper_2407_17353_amd import binding as sc

    mode = case.mode if mode is None else mode
    A = case.make_a(dev)
    B = case.make_b(dev)
    a = sc.ScaledArray(A, case.fa, sc.scale_tensor(case.a_scale_log2, dev), case.ta)
    b = sc.ScaledArray(B, case.fb, sc.scale_tensor(case.b_scale_log2, dev), case.tb)
    out = sc.empty_scaled(case.M, case.N, case.fout, dev)
    fused = act != 0 or residual_seed is not None
    # block scales keep the fp32 intermediate of the fused calls
    need = sc.scalify_matmul_workspace_size_opts(case.M, case.N, case.fout, mode,
                                                 fused or mx_seed is not None)
    if ws is None or ws.numel() < need:
        ws = sc.workspace(need, dev)
    state = torch.zeros(1, dtype=torch.float32, device=dev)
    kw = {"amax_in": state, "amax_out": state} if mode == sc.RESCALE_DELAYED else {}
    if fused:
        kw["activation"] = act
    if residual_seed is not None:
        from paper_2407_17353_amd import workloads as wl
        R = wl.fp8_normal((case.M, case.N), wl.E4M3, residual_seed, dev)
        kw["residual"] = sc.ScaledArray(R, wl.E4M3, sc.scale_tensor(1, dev))
    if mx_seed is not None:
        from paper_2407_17353_amd import workloads as wl
        # packed once, as a weight's scales would be (outside the timed calls)
        kw["a_block_scale"] = sc.scalify_mx_pack_block_scales(
            wl.mx_block_scales(case.M, case.K, mx_seed, device=dev), case.K)
        kw["b_block_scale"] = sc.scalify_mx_pack_block_scales(
            wl.mx_block_scales(case.N, case.K, mx_seed + 1, device=dev), case.K)
    stream = torch.cuda.current_stream()
    settled = None
    if settle:
        settled = settle_clock(lambda: sc.scalify_matmul(a, b, out, rescale=mode, ws=ws, **kw),
                               stream)
    for _ in range(warmup):
        sc.scalify_matmul(a, b, out, rescale=mode, ws=ws, **kw)

    def new_event():
        return torch.cuda.Event(enable_timing=True)

    # Every EVENT_EVERY-th call of the timed region is bracketed by events
    # around the GEMM kernel (an event pair costs the stream a few
    # microseconds, which would otherwise be charged to every call).
    evs = [[new_event(), new_event(), None] if k % EVENT_EVERY == 0 else None
           for k in range(steps)]
    t0, t1 = new_event(), new_event()
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t0.record(stream)
    for k in range(steps):
        sc.scalify_matmul(a, b, out, rescale=mode, ws=ws, events=evs[k], **kw)
    t1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    total_ms = t0.elapsed_time(t1)
    gemm = sorted(e[0].elapsed_time(e[1]) for e in evs if e is not None)
    gemm_ms = sum(gemm) / len(gemm)
    # Breakdown pass, outside the timed region: GEMM and epilogue both bracketed.
    nb = min(steps, 20)
    evb = [[new_event() for _ in range(3)] for _ in range(nb)]
    for k in range(nb):
        sc.scalify_matmul(a, b, out, rescale=mode, ws=ws, events=evb[k], **kw)
    torch.cuda.synchronize()
    cast_ms = sum(e[1].elapsed_time(e[2]) for e in evb) / nb

    def pct(q):
        return gemm[min(len(gemm) - 1, int(q * (len(gemm) - 1) + 0.5))]
    del A, B, a, b, out
    return {"ms_per_step": total_ms / steps, "wall_ms_per_step": wall * 1e3 / steps,
            "gemm_ms": gemm_ms, "cast_ms": cast_ms,
            "gemm_ms_p10": pct(0.1), "gemm_ms_p50": pct(0.5), "gemm_ms_p90": pct(0.9),
            "settle": settled}, ws


def time_layernorm(dev, steps, warmup, R=16384, D=4096):
    """The scaled LayerNorm of a 16384-token, d = 4096 transformer layer
    (Appendix C.2): forward FP16 -> E4M3 (scale 1) and the input gradient
    E5M2 dy, FP16 x -> E5M2 dx with the dynamic rescale (Section 4), each
    timed with HIP events over `steps` calls. Algorithmic bytes: forward
    R*D*(2 + 1); backward R*D*(2*(1 + 2) + 1): the statistic precedes the
    cast, so x and dy are read twice."""
    import torch
    from paper_2407_17353_amd import binding as sc
    from paper_2407_17353_amd import workloads as wl

    g = torch.Generator(device="cpu").manual_seed(wl.seed_of(5, 60))
    x = sc.ScaledArray((torch.randn((R, D), generator=g) * 1.5).to(torch.float16).view(torch.int16)
                       .to(dev), sc.F16, sc.scale_tensor(0, dev))
    dy = sc.ScaledArray(wl.fp8_normal((R, D), wl.E5M2, wl.seed_of(5, 61), dev), wl.E5M2,
                        sc.scale_tensor(-8, dev))
    gamma = (1.0 + 0.2 * torch.randn(D, generator=g)).to(dev)
    beta = (0.1 * torch.randn(D, generator=g)).to(dev)
    y = sc.empty_scaled(R, D, sc.E4M3, dev)
    dx = sc.empty_scaled(R, D, sc.E5M2, dev)
    dgamma = torch.empty(D, device=dev)
    dbeta = torch.empty(D, device=dev)
    ws = sc.workspace(sc.scalify_layernorm_bwd_workspace_size(R, D), dev)
    res = {}
    calls = {"fwd": lambda: sc.scalify_layernorm_fwd(x, y, gamma=gamma, beta=beta, eps=1e-5),
             "bwd": lambda: sc.scalify_layernorm_bwd(dy, x, dx, gamma=gamma, eps=1e-5,
                                                     dgamma=dgamma, dbeta=dbeta, ws=ws)}
    nbytes = {"fwd": R * D * 3, "bwd": R * D * 7}
    for name, fn in calls.items():
        for _ in range(warmup):
            fn()
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0.record()
        for _ in range(steps):
            fn()
        t1.record()
        torch.cuda.synchronize()
        us = t0.elapsed_time(t1) / steps * 1e3
        res[name] = {"us": round(us, 2), "GB/s": round(nbytes[name] / us / 1e3, 1),
                     "frac_hbm": round(nbytes[name] / us / 1e3 / PEAK_HBM_GBS, 4),
                     "alg_bytes": nbytes[name]}
    res["shape"] = [R, D]
    return res


def time_rescale(dev, steps, warmup, shapes=((8192, 8192), (16384, 16384))):
    """The standalone dynamic rescale (Section 3.3) of an fp32 matrix to E4M3:
    amax pass, power-of-two update, saturating RNE cast, timed with HIP events
    over `steps` calls per shape. Algorithmic bytes 9 per element: the
    statistic precedes the cast, so the fp32 input is read twice (8 B) and
    one E4M3 code is written."""
    import torch
    from paper_2407_17353_amd import binding as sc
    from paper_2407_17353_amd import workloads as wl

    res = {}
    for R, C in shapes:
        g = torch.Generator(device="cpu").manual_seed(wl.seed_of(4, 50))
        x = sc.ScaledArray(torch.randn((R, C), generator=g).to(dev), sc.F32, sc.scale_tensor(3, dev))
        out = sc.empty_scaled(R, C, sc.E4M3, dev)
        ws = sc.workspace(sc.scalify_rescale_workspace_size(R * C), dev)
        for _ in range(warmup):
            sc.scalify_rescale(x, out, ws=ws)
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0.record()
        for _ in range(steps):
            sc.scalify_rescale(x, out, ws=ws)
        t1.record()
        torch.cuda.synchronize()
        us = t0.elapsed_time(t1) / steps * 1e3
        nbytes = 9 * R * C
        res[f"{R}x{C}"] = {"us": round(us, 2), "GB/s": round(nbytes / us / 1e3, 1),
                           "frac_hbm": round(nbytes / us / 1e3 / PEAK_HBM_GBS, 4),
                           "alg_bytes": nbytes}
        del x, out, ws
    res["formats"] = "fp32 -> e4m3, amax rescale"
    return res


def cpu_baseline(case, target_s):
    """The oracle as it stands (fp64 accumulate + epilogue), timed on the
    first m rows of the same workload, m chosen for about target_s seconds."""
    import numpy as np
    from oracle import oracle as orc

    A = case.make_a("cuda:0").cpu().numpy()   # the very bytes the GPU run used
    B = case.make_b("cuda:0").cpu().numpy()
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))

    def run(m):
        t = time.perf_counter()
        orc.matmul(A[:m], case.fa, False, 2.0 ** case.a_scale_log2, B, case.fb, False,
                   2.0 ** case.b_scale_log2, out_fmt=case.fout)
        return time.perf_counter() - t

    m = max(1, threads)
    t = run(m)
    if t < target_s / 4:
        m = int(min(case.M, max(m, m * target_s / max(t, 1e-3))) // threads * threads) or threads
        t = run(m)
    flops = 2.0 * m * case.N * case.K
    res = {"value": flops / t / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
           "sample": f"rows 0..{m - 1} of A (a {m}x{case.N}x{case.K} scaled matmul: fp64 "
                     f"accumulation, amax rescale and cast), {t:.1f} s",
           "seconds": round(t, 2), "rows": m, "cpu_model": cpu_model()}
    res["per_config"] = oracle_per_config(threads)
    res["config1_one_core"] = oracle_config1_one_core()
    return res


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_sample(case, m):
    """Seconds of the oracle on logical rows 0..m-1 of A of one GemmCase."""
    from oracle import oracle as orc
    A = case.make_a("cpu").numpy()
    B = case.make_b("cpu").numpy()
    Asub = A[:, :m].copy() if case.ta else A[:m]
    t = time.perf_counter()
    orc.matmul(Asub, case.fa, case.ta, 2.0 ** case.a_scale_log2, B, case.fb, case.tb,
               2.0 ** case.b_scale_log2, out_fmt=case.fout)
    return time.perf_counter() - t


def oracle_per_config(threads, budget_s=1.5):
    """The oracle on the first GEMM of every configuration: a row sample
    sized for about budget_s seconds, its rate, and the whole GEMM's time
    extrapolated from it (the oracle's time is linear in the rows)."""
    from paper_2407_17353_amd import workloads as wl
    out = {}
    for cfg, cases in wl.all_configs().items():
        c = cases[0]
        m = min(c.M, max(1, threads))
        t = _oracle_sample(c, m)
        if t < budget_s / 4 and m < c.M:
            m = min(c.M, int(m * budget_s / max(t, 1e-3)))
            t = _oracle_sample(c, m)
        rate = 2.0 * m * c.N * c.K / t
        out[f"config{cfg}"] = {"gemm": c.name, "M": c.M, "N": c.N, "K": c.K, "rows": m,
                               "seconds": round(t, 3), "tflops": round(rate / 1e12, 5),
                               "whole_gemm_s_est": round(c.flops / rate, 4)}
    return out


def oracle_config1_one_core():
    """Configuration 1 (256^3) in full on one thread of the CPU."""
    import ctypes
    from paper_2407_17353_amd import workloads as wl
    c = wl.config_1()[0]
    gomp = ctypes.CDLL("libgomp.so.1")
    n0 = gomp.omp_get_max_threads()
    gomp.omp_set_num_threads(1)
    try:
        t = _oracle_sample(c, c.M)
    finally:
        gomp.omp_set_num_threads(n0)
    return {"gemm": c.name, "seconds": round(t, 4), "tflops": round(c.flops / t / 1e12, 6),
            "cores": 1}


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path "
              "(it would shard by output tiles, with one all-reduce of the amax per call)",
              file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2407_17353_amd import binding as sc
    from paper_2407_17353_amd import workloads as wl

    if not os.path.exists(sc.LIB_PATH):
        from paper_2407_17353_amd import build as hip_build
        hip_build.build()
    sc.load_library()
    dev = "cuda:0"
    if args.copy_calibration:
        copy_calibration(dev)
    case = wl.config_4(8192, wl.E4M3)[0]
    res, ws = time_case(case, args.steps, args.warmup, dev, settle=True)
    flops = case.flops
    value = flops / (res["ms_per_step"] * 1e-3) / 1e12
    gemm_tflops = flops / (res["gemm_ms"] * 1e-3) / 1e12
    line = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(res["ms_per_step"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp8e4m3",
        "data": "synthetic",
        "config": {"workload": "scaled matmul 8192x8192x8192, E4M3 x E4M3 -> E4M3, amax "
                               "rescale + saturating RNE cast (square sweep, 8192 case)",
                   "M": case.M, "N": case.N, "K": case.K, "a_fmt": "e4m3", "b_fmt": "e4m3",
                   "out_fmt": "e4m3", "layout": "A [M][K], B [K][N]",
                   "scales_log2": [case.a_scale_log2, case.b_scale_log2]},
        "pct_of_peak": round(100.0 * value / PEAK_FP8_TFLOPS, 2),
        # whole call (prologue + GEMM + cast, every launch gap) against the
        # dense FP8 peak; roofline.frac below is the GEMM kernel alone
        "frac_call": round(value / PEAK_FP8_TFLOPS, 4),
        "gemm_kernel_us": round(res["gemm_ms"] * 1e3, 2),
        "gemm_kernel_us_p10_p50_p90": [round(res[k] * 1e3, 1)
                                       for k in ("gemm_ms_p10", "gemm_ms_p50", "gemm_ms_p90")],
        "epilogue_cast_us": round(res["cast_ms"] * 1e3, 2),
        # untimed, before the warm-up calls: the call run back to back until
        # the clock has settled (the first calls of a process run slower)
        "settle": res["settle"],
        "roofline": {"bound": "mfma", "achieved": round(gemm_tflops, 2),
                     "peak": PEAK_FP8_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(gemm_tflops / PEAK_FP8_TFLOPS, 4),
                     "traffic": measured_traffic()},
    }
    # The same call forced through the single pass (one kernel: GEMM, grid
    # barrier on the statistic, cast), for comparison with the GEMM + cast
    # kernel pair timed above: 1024 tiles on one workgroup per CU, so the
    # three earlier tiles of each workgroup still pass the intermediate.
    os.environ["SCALIFY_SINGLE_PASS"] = "1"
    r2, ws = time_case(case, args.steps, args.warmup // 2, dev, ws)
    del os.environ["SCALIFY_SINGLE_PASS"]
    line["single_pass_rescale"] = {
        "value": round(flops / (r2["ms_per_step"] * 1e-3) / 1e12, 2), "unit": "TFLOP/s",
        "ms_per_step": round(r2["ms_per_step"], 4),
        "gemm_kernel_us": round(r2["gemm_ms"] * 1e3, 2),
        "epilogue_cast_us": round(r2["cast_ms"] * 1e3, 2)}
    # The delayed rescale (Section 3.3) on the same workload: the statistic of
    # the previous call sets the scale, the GEMM writes the codes directly.
    rd, ws = time_case(case, args.steps, args.warmup // 2, dev, ws, mode=sc.RESCALE_DELAYED)
    line["delayed_rescale"] = {
        "value": round(flops / (rd["ms_per_step"] * 1e-3) / 1e12, 2), "unit": "TFLOP/s",
        "ms_per_step": round(rd["ms_per_step"], 4),
        "pct_of_peak": round(100.0 * flops / (rd["ms_per_step"] * 1e-3) / 1e12 / PEAK_FP8_TFLOPS, 2),
        "gemm_kernel_us": round(rd["gemm_ms"] * 1e3, 2)}
    # The same workload with the scaled add of a residual and GELU fused into
    # the epilogue (Algorithm 3 add rule, Appendix C.1), dynamic and delayed.
    line["fused_add_gelu"] = {}
    for name, m in (("amax", sc.RESCALE_AMAX), ("delayed", sc.RESCALE_DELAYED)):
        rf, ws = time_case(case, args.steps // 2, args.warmup // 2, dev, ws, mode=m,
                           act=sc.ACT_GELU_TANH, residual_seed=wl.seed_of(4, 30))
        line["fused_add_gelu"][name] = {
            "value": round(flops / (rf["ms_per_step"] * 1e-3) / 1e12, 2), "unit": "TFLOP/s",
            "ms_per_step": round(rf["ms_per_step"], 4),
            "gemm_kernel_us": round(rf["gemm_ms"] * 1e3, 2),
            "epilogue_cast_us": round(rf["cast_ms"] * 1e3, 2) if m == sc.RESCALE_AMAX else None}
    # The same workload with MX block scales (Section 2: block-scaling formats
    # as scales broadcastable to the data), applied by the scaled MFMA.
    line["mx_block_scales"] = {}
    for name, m in (("amax", sc.RESCALE_AMAX), ("delayed", sc.RESCALE_DELAYED)):
        rm, ws = time_case(case, args.steps // 2, args.warmup // 2, dev, ws, mode=m,
                           mx_seed=wl.seed_of(4, 40))
        line["mx_block_scales"][name] = {
            "value": round(flops / (rm["ms_per_step"] * 1e-3) / 1e12, 2), "unit": "TFLOP/s",
            "ms_per_step": round(rm["ms_per_step"], 4),
            "gemm_kernel_us": round(rm["gemm_ms"] * 1e3, 2),
            "epilogue_cast_us": round(rm["cast_ms"] * 1e3, 2) if m == sc.RESCALE_AMAX else None}
    line["layernorm"] = time_layernorm(dev, 20, 10)
    line["rescale"] = time_rescale(dev, 20, 10)
    if args.sweep:
        sweep = []
        for cfg, cases in wl.all_configs().items():
            for c in cases:
                r, ws = time_case(c, max(5, args.steps // 5), 20, dev, ws)
                tf = c.flops / (r["ms_per_step"] * 1e-3) / 1e12
                row = {"config": cfg, "name": c.name, "M": c.M, "N": c.N, "K": c.K,
                       "us": round(r["ms_per_step"] * 1e3, 1), "tflops": round(tf, 1),
                       "pct_peak": round(100 * tf / PEAK_FP8_TFLOPS, 1),
                       "gemm_us": round(r["gemm_ms"] * 1e3, 1),
                       "cast_us": round(r["cast_ms"] * 1e3, 1)}
                sweep.append(row)
                print(json.dumps(row), file=sys.stderr, flush=True)
        os.makedirs(os.path.join(ROOT, "gpurun_out"), exist_ok=True)
        with open(os.path.join(ROOT, "gpurun_out", "sweep.json"), "w") as f:
            json.dump(sweep, f, indent=1)
    del ws
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(case, args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
