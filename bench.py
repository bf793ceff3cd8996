"""Benchmark of the SFDA hot path on one MI355X.

A step is one sfda_chunk_fwd call over the bf16 workload B=8, H=16, T=4096, m=64 complex
key channels (d_k=128), n=64 complex value columns (d_v=128), C=64: chunk factors, Gram
matrices, triangular solve, intra-chunk readout, state update and the chunk-to-chunk state
scan, all in one launch.  Inputs are resident in HBM before timing starts.  Throughput is
B*T tokens (every token through all H heads) per second.

Also reported on the same JSON line:
  roofline      the chunk kernel against HBM bandwidth (algorithmic bytes / launch time),
                with achieved MFMA rates (useful causal flops, dense-tile flops and the
                executed matrix-core flops counted by SQ_INSTS_VALU_MFMA_MOPS_BF16) beside it
  decode        the sfda_step kernel on the state [512, 32, 64, 64] complex fp32 (HBM-bound)
  launch_ms     mean (= ms_per_step), median, minimum and maximum of the K per-launch
                intervals between HIP events recorded on the launch stream
  launch_ms_c128  the same statistics for the same call with C = 128 (K launches after W)
  cpu_baseline  the CPU oracle (complex128 recurrence) on a bounded sample of the workload,
                on every host thread and on one thread, with the CPU model
Each kernel runs an untimed settle phase (about 0.3 s of launches) before its W warm-up
and K timed launches: the GPU's clocks drop while the host generates the next workload's
inputs, and a short run (the driver's 20 steps after 5) would otherwise time the ramp.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--only chunk|decode]
       [--no-cpu-baseline] [--mode copy|rmw|long|gated|bwd|dec|f32]   (copy: a plain device copy, for counter
       scaling; rmw: an in-place pass over 1 GiB, the decode step's access pattern; long:
       the long-context workload, one workgroup per head against the segment-parallel scan;
       gated: the benchmarked shape through sfda_chunk_fwd_gated; bwd: sfda_chunk_bwd on the
       benchmarked shape and on the float32 workload B=4, H=8, T=2048; dec: the write-decoupled
       variant on the benchmarked batch, heads and length (C=64, run as 16-token chunks); f32: the float32
       workload B=4, H=8, T=2048 against the fp32 matrix-core peak: the plain launch,
       value-column slices and segment-parallel)
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "SFDA fwd tokens/s (H=16,d_k=128,d_v=128,T=4096,C=64) + % MFMA/HBM peak"
HBM_PEAK_GBS = 8000.0
BF16_MFMA_PEAK_TFLOPS = 2516.6
PROFILES = os.path.join(ROOT, "profiles")
# the sources of the kernels the default bench line times (the bf16 chunk kernel and the
# decode step); a counter summary is used only while they are unchanged
KERNEL_SOURCES = ["paper_2607_11897_amd/csrc/sfda_chunk_bf16.hip", "paper_2607_11897_amd/csrc/sfda_step.hip",
                  "paper_2607_11897_amd/csrc/sfda_device.h"]
FP32_MFMA_PEAK_TFLOPS = 157.3
SETTLE_S = 0.3


KERNEL_BLOCK = 16       # tokens per block of the bf16 chunk kernel's factorisation


def kernel_hash() -> str:
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def chunk_bytes_per_token_head(m, n, T, in_bytes, out_bytes):
    """Algorithmic HBM bytes per token and head: q, k (m complex), v (n complex), alpha,
    theta (m real), beta, o (n complex) once each, plus S0 and S_T (m x n complex fp32)
    amortised over the T tokens of a head."""
    return (2 * m * 2 + n * 2 + 2 * m + 1) * in_bytes + n * 2 * out_bytes + 2 * m * n * 8 / T


def chunk_flops_per_chunk_head(C, m, n):
    """Real flops per chunk and head (a complex multiply-add is 8 real flops).
    useful: Gram L' and A (causal halves, C^2 m / 2 each), Wt and U (C^2 m / 2, C^2 n / 2),
    A Delta (C^2 n / 2), Wt S, conj(Q)G S and the state update (C m n each), and the
    triangular solve (C^3 / 6).  dense_tile: the same eight products counted as full
    tiles, without the solve."""
    useful = 8 * (C * C * (3 * m + 2 * n) / 2 + 3 * C * m * n + C ** 3 / 6)
    tile = 8 * (C * C * (3 * m + 2 * n) + 3 * C * m * n)
    return useful, tile


def decode_bytes_per_head(m, n, in_bytes=4, out_bytes=4):
    """State read and written once (m x n complex fp32 each way) plus one token's q, k, v,
    alpha, theta, beta and o."""
    return 2 * m * n * 8 + (2 * m * 2 + n * 2 + 2 * m + 1) * in_bytes + n * 2 * out_bytes


def load_traffic(kernel: str, workload: str):
    """HBM traffic measured by counters for a kernel, if a committed counter summary exists
    for the current kernel source."""
    path = os.path.join(PROFILES, f"{kernel}_{workload}_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)
    if d.get("kernel_hash") != kernel_hash():
        return None
    return d.get("bytes_per_launch")


def load_mfma_counters(kernel: str, workload: str):
    """Executed matrix-core flops per launch, from a committed counter summary
    (SQ_INSTS_VALU_MFMA_MOPS_BF16) for the current kernel source, or None."""
    path = os.path.join(PROFILES, f"{kernel}_{workload}_mfma.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)
    if d.get("kernel_hash") != kernel_hash():
        return None
    return d.get("mfma_flops_per_launch")


def timed_stats(fn, steps, warmup, stream):
    """W untimed launches, then exactly K launches with a HIP event recorded on the launch
    stream before the first and after every launch.  Returns the mean over the whole
    bracketed region (total / K, the ms_per_step of the bench line) and the median,
    minimum and maximum of the per-launch event intervals, in ms."""
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    evs[0].record(stream)
    for i in range(steps):
        fn()
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    per = sorted(evs[i].elapsed_time(evs[i + 1]) for i in range(steps))
    mid = steps // 2
    median = per[mid] if steps % 2 else 0.5 * (per[mid - 1] + per[mid])
    return {"mean": evs[0].elapsed_time(evs[-1]) / steps, "median": median, "min": per[0],
            "max": per[-1]}


def timed(fn, steps, warmup, stream):
    return timed_stats(fn, steps, warmup, stream)["mean"]   # ms per call


def settle_clocks(fn, seconds, stream):
    """Untimed launches of fn for about `seconds` of wall time (the GPU's clocks ramp up
    over the first tens of milliseconds of work after it has been idle)."""
    import torch
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(20):
            fn()
        torch.cuda.synchronize()


def bench_chunk(args, stream):
    import numpy as np
    import torch
    from paper_2607_11897_amd import inputs as I
    from paper_2607_11897_amd import sfda
    w = I.WORKLOADS["fwd_bf16_b8h16_t4k"]
    print(f"# generating inputs for {w.name}", file=sys.stderr, flush=True)
    x = I.make_chunk_inputs(w)
    st = x.storage()
    dev = torch.device("cuda:0")

    def up(a, dt):
        if dt == "bf16":
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)

    d = {k: up(st[k], w.dtype) for k in ("q", "k", "v", "alpha", "theta", "beta")}
    S0 = up(st["S0"], "f32")
    B, H, T, m, n = x.shape
    o = torch.empty((B, H, T, n, 2), dtype=torch.bfloat16, device=dev)
    S_T = torch.empty((B, H, m, n, 2), dtype=torch.float32, device=dev)

    def run():
        sfda.chunk_fwd(d["q"], d["k"], d["v"], d["alpha"], d["theta"], d["beta"], S0, C=w.C,
                       o=o, S_T=S_T, segments=None, stream=stream)

    print(f"# timing sfda_chunk_fwd: {SETTLE_S} s of untimed launches, warmup {args.warmup}, "
          f"steps {args.steps}", file=sys.stderr, flush=True)
    settle_clocks(run, SETTLE_S, stream)
    stats = timed_stats(run, args.steps, args.warmup, stream)
    ms = stats["mean"]

    # the same launch with C = 128 (the kernel's 16-token blocking does not depend on C, and
    # neither does the result: Thm 6.1), reported beside the C = 64 line
    def run128():
        sfda.chunk_fwd(d["q"], d["k"], d["v"], d["alpha"], d["theta"], d["beta"], S0, C=128,
                       o=o, S_T=S_T, segments=None, stream=stream)

    stats128 = timed_stats(run128, args.steps, args.warmup, stream)
    units = B * H * T
    bytes_alg = chunk_bytes_per_token_head(m, n, T, 2, 2) * units
    # the kernel evaluates 16-token blocks whatever C is (the result does not depend on C):
    # its flops are those of 16-token chunks
    useful, tile = chunk_flops_per_chunk_head(KERNEL_BLOCK, m, n)
    nchunk = B * H * (T // KERNEL_BLOCK)
    sec = ms / 1e3
    achieved = bytes_alg / sec / 1e9
    traffic = load_traffic("chunk_fwd", w.name)
    exec_flops = load_mfma_counters("chunk_fwd", w.name)
    return dict(
        w=w, ms=ms, tokens_per_s=B * T / sec, x=x,
        launch_ms={k: round(v, 4) for k, v in stats.items()},
        launch_ms_c128={k: round(v, 4) for k, v in stats128.items()},
        roofline={"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS,
                  "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                  "traffic": traffic,
                  "kernel": "sfda::pipe::chunk_pipe_kernel<bf16 out> (C=64, two workgroups per head)",
                  "bytes_per_launch": int(bytes_alg),
                  "bytes_per_token_head": chunk_bytes_per_token_head(m, n, T, 2, 2),
                  "mfma": {"peak_tflops": BF16_MFMA_PEAK_TFLOPS,
                           "useful_tflops": round(useful * nchunk / sec / 1e12, 2),
                           "useful_frac": round(useful * nchunk / sec / 1e12 / BF16_MFMA_PEAK_TFLOPS, 4),
                           "tile_tflops": round(tile * nchunk / sec / 1e12, 2),
                           "tile_frac": round(tile * nchunk / sec / 1e12 / BF16_MFMA_PEAK_TFLOPS, 4),
                           "exec_tflops": None if exec_flops is None else round(exec_flops / sec / 1e12, 2),
                           "exec_frac": None if exec_flops is None
                           else round(exec_flops / sec / 1e12 / BF16_MFMA_PEAK_TFLOPS, 4),
                           "flops_per_chunk_head": {"useful": useful, "tile": tile,
                                                    "exec": None if exec_flops is None
                                                    else exec_flops / nchunk}}},
    )


def bench_decode(args, stream):
    import torch
    from paper_2607_11897_amd import inputs as I
    from paper_2607_11897_amd import sfda
    D = I.DECODE
    B, H, m, n = D["B"], D["H"], D["m"], D["n"]
    gen = torch.Generator(device="cuda")
    gen.manual_seed(D["seed"])
    S = torch.randn(B, H, m, n, 2, generator=gen, device="cuda") * 0.0707
    q, k, v, a, th, bt = I.fill_decode_bulk_torch(gen, B, H, m, n, "cuda")
    o = torch.empty((B, H, n, 2), device="cuda")

    def run():
        sfda.step(q, k, v, a, th, bt, S, o=o, stream=stream)

    steps = max(20, args.steps)
    print(f"# timing sfda_step: {SETTLE_S} s of untimed steps, then {steps} steps", file=sys.stderr, flush=True)
    settle_clocks(run, SETTLE_S, stream)
    stats = timed_stats(run, steps, max(3, args.warmup), stream)
    ms = stats["mean"]
    bytes_step = decode_bytes_per_head(m, n) * B * H
    gbs = bytes_step / (ms / 1e3) / 1e9
    return {"workload": D["name"], "us_per_step": round(ms * 1e3, 2),
            "launch_us": {k: round(v * 1e3, 2) for k, v in stats.items()},
            "tokens_per_s": round(B / (ms / 1e3), 1),
            "roofline": {"bound": "hbm", "achieved": round(gbs, 2), "peak": HBM_PEAK_GBS,
                         "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4),
                         "traffic": load_traffic("step", D["name"]),
                         "kernel": "sfda::step_pair_kernel<f32, 64>",
                         "bytes_per_launch": int(bytes_step)}}


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(x, budget_s=12.0, single_budget_s=6.0):
    """The oracle on whole batch elements of the workload (all H heads, all T tokens), one
    after another -- passing over the batch again if it finishes early -- until about
    budget_s seconds have been spent, on every host thread; then the same on one thread
    for about single_budget_s seconds."""
    import oracle
    B, H, T, m, n = x.shape

    def run(nthreads, budget):
        done = 0
        t0 = time.perf_counter()
        while True:
            b = done % B
            oracle.recurrence(x.q[b:b + 1], x.k[b:b + 1], x.v[b:b + 1], x.alpha[b:b + 1],
                              x.theta[b:b + 1], x.beta[b:b + 1],
                              None if x.S0 is None else x.S0[b:b + 1], nthreads=nthreads)
            done += 1
            if time.perf_counter() - t0 >= budget:
                break
        return done, time.perf_counter() - t0

    threads = oracle.max_threads()
    done, el = run(0, budget_s)
    done1, el1 = run(1, single_budget_s)
    return {"value": round(done * T / el, 1), "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"{done} batch elements of {B} (taken in turn) x {H} heads x {T} tokens "
                      f"(complex128 recurrence), {el:.1f} s",
            "cpu_model": cpu_model(),
            "single_thread": {"value": round(done1 * T / el1, 1), "unit": "tokens/s", "cores": 1,
                              "sample": f"{done1} batch elements x {H} heads x {T} tokens, {el1:.1f} s"}}


def cpu_baseline_backward(x, dO, dS, budget_s=10.0):
    """The oracle's reverse-mode sweep (oracle.backward, complex128 numpy) on whole heads of
    the workload, one after another, until about budget_s seconds have been spent; the
    rate counts a token as one position through all H heads, like the GPU figure."""
    from oracle import backward as BW
    B, H, T, m, n = x.shape
    done = 0
    t0 = time.perf_counter()
    while True:
        b, h = divmod(done % (B * H), H)
        BW.recurrence_backward(x.q[b:b + 1, h:h + 1], x.k[b:b + 1, h:h + 1], x.v[b:b + 1, h:h + 1],
                               x.alpha[b:b + 1, h:h + 1], x.theta[b:b + 1, h:h + 1], x.beta[b:b + 1, h:h + 1],
                               None if x.S0 is None else x.S0[b:b + 1, h:h + 1], dO[b:b + 1, h:h + 1],
                               dS[b:b + 1, h:h + 1])
        done += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    el = time.perf_counter() - t0
    return {"value": round(done * T / H / el, 1), "unit": "tokens/s", "cores": 1, "kind": "oracle",
            "sample": f"{done} heads of {B * H} (taken in turn) x {T} tokens (complex128 reverse sweep, "
                      f"numpy in one process), {el:.1f} s"}


def long_context(args):
    """The long-context float32 workload (B=1, H=16, T=65536, m=n=64, C=64): one
    sfda_chunk_fwd launch (one workgroup per head) against sfda_chunk_fwd_segmented with
    G segments per head (the scan split G ways, joined by the affine segment law)."""
    import numpy as np
    import torch
    from paper_2607_11897_amd import inputs as I
    from paper_2607_11897_amd import sfda
    w = I.WORKLOADS["long_f32_h16_t64k"]
    print(f"# generating inputs for {w.name}", file=sys.stderr, flush=True)
    x = I.make_chunk_inputs(w)
    st = x.storage()
    d = {k: torch.from_numpy(np.ascontiguousarray(st[k], dtype=np.float32)).cuda()
         for k in ("q", "k", "v", "alpha", "theta", "beta")}
    S0 = torch.from_numpy(np.ascontiguousarray(st["S0"], dtype=np.float32)).cuda()
    B, H, T, m, n = x.shape
    o = torch.empty((B, H, T, n, 2), dtype=torch.float32, device="cuda")
    S_T = torch.empty((B, H, m, n, 2), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    out = {"mode": "long", "workload": w.name, "B": B, "H": H, "T": T, "m": m, "n": n, "C": w.C,
           "dtype": "f32", "ms": {}, "tokens_per_s": {}}
    # the workload's chunk length, and C = 16 (the same result to rounding; the fp32 kernel
    # runs two waves per SIMD at C <= 32)
    for C, Gs in ((w.C, (None, 4, 8, 16, 32, "auto")), (16, (None, 16))):
        for G in Gs:
            ws = None if G in (None, "auto") else torch.empty(sfda.segmented_workspace_bytes(B, H, T, m, n, G),
                                                              dtype=torch.uint8, device="cuda")

            def run():
                sfda.chunk_fwd(d["q"], d["k"], d["v"], d["alpha"], d["theta"], d["beta"], S0, C=C,
                               o=o, S_T=S_T, segments=G, workspace=ws, stream=stream)

            key = ("plain" if G is None else "auto" if G == "auto" else f"segments_{G}") + ("" if C == w.C else f"_C{C}")
            print(f"# timing {key}", file=sys.stderr, flush=True)
            ms = timed(run, 3 if G is None else 10, 1, stream)
            out["ms"][key] = round(ms, 3)
            out["tokens_per_s"][key] = round(B * T / (ms / 1e3), 1)
    out["kernel_hash_fp32_path"] = bwd_hash()
    print(json.dumps(out), flush=True)


def fp32_forward(args):
    """The float32 workload (B=4, H=8, T=2048, m=n=64, C=64) through the fp32 chunk kernel,
    against the fp32 matrix-core peak (its roofline bound: 72 flop per byte against an fp32
    ridge of 20): one workgroup per head at the workload's C = 64 and at C = 16 and 32 (the
    same result to rounding), and sfda_chunk_fwd_segmented with G segments per head (32
    heads leave most of the 256 CUs idle).  Useful flops are the method's (causal halves,
    solve included) for the whole result, whatever the path; the oracle is timed beside it.
    slice: value columns per workgroup (sfda_chunk_fwd_sliced: 64 / slice workgroups per
    head, each repeating the head's chunk factors)."""
    import numpy as np
    import torch
    from paper_2607_11897_amd import inputs as I
    from paper_2607_11897_amd import sfda
    w = I.WORKLOADS["fwd_f32_b4h8_t2k"]
    print(f"# generating inputs for {w.name}", file=sys.stderr, flush=True)
    x = I.make_chunk_inputs(w)
    st = x.storage()
    d = {k: torch.from_numpy(np.ascontiguousarray(st[k], dtype=np.float32)).cuda()
         for k in ("q", "k", "v", "alpha", "theta", "beta")}
    S0 = torch.from_numpy(np.ascontiguousarray(st["S0"], dtype=np.float32)).cuda()
    B, H, T, m, n = x.shape
    o = torch.empty((B, H, T, n, 2), dtype=torch.float32, device="cuda")
    S_T = torch.empty((B, H, m, n, 2), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    # the kernel evaluates 16-token blocks whatever C is (the result does not depend on C):
    # its flops are those of 16-token chunks
    useful, tile = chunk_flops_per_chunk_head(KERNEL_BLOCK, m, n)
    nchunk = B * H * (T // KERNEL_BLOCK)
    bytes_alg = chunk_bytes_per_token_head(m, n, T, 4, 4) * B * H * T
    runs = []
    # (every C runs 16-token chunks: slices and segments are the knobs that change the launch)
    # ("auto": the binding's default, the segment count sfda_chunk_fwd_auto_segments picks)
    for C, G, sl in ((64, None, None), (64, None, 32), (64, None, 16), (64, None, 8),
                     (64, 4, None), (64, 8, None), (64, 16, None), (64, "auto", None)):
        ws = None if G in (None, "auto") else torch.empty(sfda.segmented_workspace_bytes(B, H, T, m, n, G),
                                                          dtype=torch.uint8, device="cuda")

        def run():
            sfda.chunk_fwd(d["q"], d["k"], d["v"], d["alpha"], d["theta"], d["beta"], S0, C=C,
                           o=o, S_T=S_T, slice=sl, segments=G, workspace=ws, stream=stream)

        print(f"# timing C={C} G={G} slice={sl}", file=sys.stderr, flush=True)
        ms = timed(run, args.steps, min(args.warmup, 10), stream)
        sec = ms / 1e3
        tf = useful * nchunk / sec / 1e12
        runs.append({"C": C, "segments": G, "slice": sl, "ms": round(ms, 4),
                     **({"auto_segments": sfda.auto_segments(B, H, T, m, n, C)} if G == "auto" else {}),
                     "tokens_per_s": round(B * T / sec, 1),
                     "roofline": {"bound": "mfma", "achieved": round(tf, 2), "peak": FP32_MFMA_PEAK_TFLOPS,
                                  "unit": "TFLOP/s", "frac": round(tf / FP32_MFMA_PEAK_TFLOPS, 4),
                                  "traffic": None,
                                  "tile_tflops": round(tile * nchunk / sec / 1e12, 2)},
                     "hbm_GBps_algorithmic": round(bytes_alg / sec / 1e9, 1)})
        del ws
    out = {"mode": "f32", "workload": w.name, "B": B, "H": H, "T": T, "m": m, "n": n, "C": w.C,
           "dtype": "f32", "flops_per_chunk_head": {"useful": useful, "tile": tile},
           "bytes_per_token_head": chunk_bytes_per_token_head(m, n, T, 4, 4), "runs": runs,
           "kernel_hash_fp32_path": bwd_hash()}
    if not args.no_cpu_baseline:
        print("# timing the CPU oracle", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(x)
    print(json.dumps(out), flush=True)


def gated(args):
    """The benchmarked shape (bf16, B=8, H=16, T=4096, m=n=64, C=64) on pre-activations:
    sfda_chunk_fwd_gated, alpha, theta, beta and the key normalisation formed inside the
    kernel (compare with the default bench line, sfda_chunk_fwd on the same sizes)."""
    import torch
    from paper_2607_11897_amd import inputs as I
    from paper_2607_11897_amd import sfda
    B, H, T, m, n, C = 8, 16, 4096, 64, 64, 64
    print("# generating gated inputs", file=sys.stderr, flush=True)
    g = I.make_gated_inputs(B, H, T, m, n, "bf16", seed=2002)
    st = g.storage()
    import numpy as np
    up = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(torch.bfloat16)
    d = {k: up(st[k]) for k in ("q", "k_raw", "v", "a", "b", "c")}
    S0 = torch.from_numpy(np.ascontiguousarray(st["S0"], dtype=np.float32)).cuda()
    o = torch.empty((B, H, T, n, 2), dtype=torch.bfloat16, device="cuda")
    S_T = torch.empty((B, H, m, n, 2), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    gp = dict(alpha_min=0.9, alpha_max=1.0, theta_max=0.5, eps=1e-6)

    def run_gated():
        sfda.chunk_fwd_gated(d["q"], d["k_raw"], d["v"], d["a"], d["b"], d["c"], S0, C=C, o=o,
                             S_T=S_T, stream=stream, **gp)

    ms_g = timed(run_gated, args.steps, args.warmup, stream)
    out = {"mode": "gated", "workload": "gated_bf16_b8h16_t4k", "B": B, "H": H, "T": T, "m": m,
           "n": n, "C": C, "gates": gp, "ms_gated": round(ms_g, 4),
           "tokens_per_s_gated": round(B * T / (ms_g / 1e3), 1), "kernel_hash": kernel_hash()}
    print(json.dumps(out), flush=True)


def bwd_flops_per_chunk_head(C, m, n):
    """Real flops per chunk and head of sfda_chunk_bwd's three passes, causal halves counted
    (a complex multiply-add is 8 real flops; X = C m n, Y = C^2 m / 2, Z = C^2 n / 2):
    forward scan L' Y, solve C^3/6, T conj(V) Z, T (conj(K) G) Y, Wt S X, state update X;
    adjoint scan L', A 2Y, solve C^3/6, conj(Y') G X, A^* G_R Z, N^* G_Delta Z, two state
    products 2X; gradient pass L' Y, E X, L' Delta Z, G_A and G_N 2Z, G_Yp, G_R S^*,
    G_E S^* 3X, four token products with conj(K/G), conj(conj(K)G), conj(conj(Q)G) 4Y."""
    X, Y, Z = C * m * n, C * C * m / 2, C * C * n / 2
    fwd = Y + C ** 3 / 6 + Z + Y + 2 * X
    adj = 2 * Y + C ** 3 / 6 + X + 2 * Z + 2 * X
    grd = Y + X + Z + 2 * Z + 3 * X + 4 * Y
    return 8 * (fwd + adj + grd)


def bwd_bytes_per_token_head(m, n, in_bytes, out_bytes):
    """Algorithmic HBM bytes of the backward per token and head: the forward's inputs read
    once, dL/do read once, every input gradient written once (state terms are amortised
    over T and left out)."""
    inputs = (2 * m * 2 + n * 2 + 2 * m + 1) * in_bytes
    return inputs + n * 2 * out_bytes + inputs


def backward(args):
    """sfda_chunk_bwd (three launches: recording forward scan, adjoint scan, gradient pass)
    on the benchmarked shape (bf16) and on the float32 workload B=4, H=8, T=2048, inputs and
    upstream gradients resident in HBM."""
    import torch
    from paper_2607_11897_amd import inputs as I
    from paper_2607_11897_amd import sfda
    import numpy as np
    # the backward runs 16-token chunks whatever C it is given (the gradients do not depend
    # on the chunk length, to rounding; 16 keeps 1 / g in range for strong decay)
    C_BWD = 16
    res = {"mode": "bwd", "kernel_hash_bwd": bwd_hash(), "C_bwd": C_BWD, "runs": []}
    for name in ("fwd_bf16_b8h16_t4k", "fwd_f32_b4h8_t2k"):
        w = I.WORKLOADS[name]
        print(f"# generating inputs for {w.name}", file=sys.stderr, flush=True)
        x = I.make_chunk_inputs(w)
        dO, dS = I.make_cotangents(w.B, w.H, w.T, w.m, w.n, w.dtype, seed=w.seed + 77)
        st = x.storage()

        def up(a, dt):
            if dt == "bf16":
                return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(torch.bfloat16)
            return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()

        d = {k: up(st[k], w.dtype) for k in ("q", "k", "v", "alpha", "theta", "beta")}
        S0 = up(st["S0"], "f32")
        dO_t = up(I.to_storage(dO, w.dtype), w.dtype)
        dS_t = up(I.to_storage(dS, "f32"), "f32")
        B, H, T, m, n = x.shape
        ws = torch.empty(sfda.bwd_workspace_bytes(B, H, T, m, n, C_BWD), dtype=torch.uint8, device="cuda")
        stream = torch.cuda.current_stream()

        def run():
            sfda.chunk_bwd(d["q"], d["k"], d["v"], d["alpha"], d["theta"], d["beta"], S0, dO_t, dS_t,
                           C=C_BWD, workspace=ws, stream=stream)

        def run_fwd():
            sfda.chunk_fwd(d["q"], d["k"], d["v"], d["alpha"], d["theta"], d["beta"], S0, C=w.C,
                           segments=None, stream=stream)

        print(f"# timing sfda_chunk_bwd on {w.name}", file=sys.stderr, flush=True)
        ms = timed(run, max(5, args.steps // 5), max(2, args.warmup // 5), stream)
        ms_f = timed(run_fwd, max(5, args.steps // 5), max(2, args.warmup // 5), stream)
        chunks = B * H * ((T + C_BWD - 1) // C_BWD)
        flops = bwd_flops_per_chunk_head(C_BWD, m, n) * chunks
        eb = 2 if w.dtype == "bf16" else 4
        nbytes = bwd_bytes_per_token_head(m, n, eb, eb) * B * H * T
        tflops = flops / (ms / 1e3) / 1e12
        peak = BF16_MFMA_PEAK_TFLOPS if w.dtype == "bf16" else FP32_MFMA_PEAK_TFLOPS
        run = {
            "workload": w.name, "B": B, "H": H, "T": T, "m": m, "n": n, "C_fwd": w.C, "C_bwd": C_BWD, "dtype": w.dtype,
            "ms_bwd": round(ms, 4), "ms_fwd": round(ms_f, 4), "bwd_over_fwd": round(ms / ms_f, 2),
            "tokens_per_s_bwd": round(B * T / (ms / 1e3), 1),
            # the whole pass against the matrix cores of the operand type it runs on, and its
            # algorithmic bytes against HBM
            "roofline": {"bound": "mfma", "achieved": round(tflops, 2), "peak": peak, "unit": "TFLOP/s",
                         "frac": round(tflops / peak, 4), "traffic": None,
                         "flops_per_chunk_head": bwd_flops_per_chunk_head(C_BWD, m, n)},
            "hbm": {"achieved_GBps": round(nbytes / (ms / 1e3) / 1e9, 1), "peak_GBps": HBM_PEAK_GBS,
                    "bytes_per_token_head": bwd_bytes_per_token_head(m, n, eb, eb)},
            "workspace_bytes": int(ws.numel())}
        if not args.no_cpu_baseline:
            print(f"# oracle backward on the CPU ({w.name})", file=sys.stderr, flush=True)
            run["cpu_baseline"] = cpu_baseline_backward(x, dO, dS)
        res["runs"].append(run)
        del d, dO_t, dS_t, ws
        torch.cuda.empty_cache()
    print(json.dumps(res), flush=True)


def dec_flops_per_chunk_head(C, m, n):
    """Real flops per chunk and head of the write-decoupled forward, causal halves counted:
    Gram blocks L'_kk, A_qk, L'_kr, A_qr (4 C^2 m / 2), Wt = T conj(K)G (C^2 m / 2), the solve
    C^3 / 6, Y = L'_kr Delta_r and T Y (2 C^2 n / 2), A_qk Delta_k and A_qr Delta_r (2 C^2 n / 2),
    Wt S, conj(Q)G S and the two state products (4 C m n)."""
    return 8 * (5 * C * C * m / 2 + 4 * C * C * n / 2 + 4 * C * m * n + C ** 3 / 6)


def decoupled(args):
    """sfda_chunk_fwd_decoupled on the benchmarked batch, heads and length (bf16, C = 64, which
    the kernel runs as 16-token chunks), beside sfda_chunk_fwd on the same sizes."""
    import numpy as np
    import torch
    from paper_2607_11897_amd import inputs as I
    from paper_2607_11897_amd import sfda
    B, H, T, m, n, C = 8, 16, 4096, 64, 64, 64
    C_RUN = 16           # the chunk length the write-decoupled kernel runs for every C
    print("# generating write-decoupled inputs", file=sys.stderr, flush=True)
    x = I.make_decoupled_inputs(B, H, T, m, n, "bf16", seed=3003)
    st = x.storage()
    up = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(torch.bfloat16)
    d = {k: up(st[k]) for k in ("q", "k", "r", "v", "alpha", "theta", "eta", "beta")}
    S0 = torch.from_numpy(np.ascontiguousarray(st["S0"], dtype=np.float32)).cuda()
    o = torch.empty((B, H, T, n, 2), dtype=torch.bfloat16, device="cuda")
    S_T = torch.empty((B, H, m, n, 2), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()

    def run_dec():
        sfda.chunk_fwd_decoupled(d["q"], d["k"], d["r"], d["v"], d["alpha"], d["theta"], d["eta"], d["beta"],
                                 S0, C=C, o=o, S_T=S_T, stream=stream)

    def run_tied():
        sfda.chunk_fwd(d["q"], d["k"], d["v"], d["alpha"], d["theta"], d["beta"], S0, C=C, o=o, S_T=S_T,
                       segments=None, stream=stream)

    ms_d = timed(run_dec, max(5, args.steps // 5), max(2, args.warmup // 5), stream)
    ms_t = timed(run_tied, max(5, args.steps // 5), max(2, args.warmup // 5), stream)
    flops = dec_flops_per_chunk_head(C_RUN, m, n) * B * H * (T // C_RUN)
    tflops = flops / (ms_d / 1e3) / 1e12
    out = {"mode": "dec", "workload": "decoupled_bf16_b8h16_t4k", "B": B, "H": H, "T": T, "m": m, "n": n,
           "C": C, "C_run": C_RUN, "ms_decoupled": round(ms_d, 4), "ms_tied_same_C": round(ms_t, 4),
           "tokens_per_s_decoupled": round(B * T / (ms_d / 1e3), 1),
           "roofline": {"bound": "mfma", "achieved": round(tflops, 2), "peak": BF16_MFMA_PEAK_TFLOPS,
                        "unit": "TFLOP/s", "frac": round(tflops / BF16_MFMA_PEAK_TFLOPS, 4), "traffic": None,
                        "flops_per_chunk_head": dec_flops_per_chunk_head(C_RUN, m, n)},
           "kernel_hash_fp32_path": bwd_hash()}
    if not args.no_cpu_baseline:
        from oracle import decoupled as Dd
        print("# oracle (write-decoupled recurrence) on the CPU", file=sys.stderr, flush=True)
        done, t0 = 0, time.perf_counter()
        while True:
            b = done % B
            Dd.decoupled_recurrence(*(getattr(x, nm)[b:b + 1] for nm in ("q", "k", "r", "v", "alpha", "theta", "eta", "beta")),
                                    x.S0[b:b + 1])
            done += 1
            if time.perf_counter() - t0 >= 10.0:
                break
        el = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": round(done * T / el, 1), "unit": "tokens/s", "cores": 1, "kind": "oracle",
                               "sample": f"{done} batch elements of {B} (taken in turn) x {H} heads x {T} tokens "
                                         f"(complex128 numpy recurrence in one process), {el:.1f} s"}
    print(json.dumps(out), flush=True)


def bwd_hash() -> str:
    h = hashlib.sha256()
    for p in ("paper_2607_11897_amd/csrc/sfda_chunk.hip", "paper_2607_11897_amd/csrc/sfda_chunk_grad.hip",
              "paper_2607_11897_amd/csrc/sfda_chunk_common.h", "paper_2607_11897_amd/csrc/sfda_device.h"):
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def copy_calibration(args):
    """A plain device-to-device copy of 1 GiB, repeated, for scaling HBM counters."""
    import torch
    nbytes = 1 << 30
    src = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    ms = timed(lambda: dst.copy_(src), max(5, args.steps), 2, torch.cuda.current_stream())
    print(json.dumps({"mode": "copy", "bytes_read": nbytes, "bytes_written": nbytes,
                      "ms_per_copy": ms, "GBps": 2 * nbytes / (ms / 1e3) / 1e9}), flush=True)


def rmw_calibration(args):
    """An in-place scaling of a 1 GiB fp32 tensor (read and write of the same bytes, the
    access pattern of the decode step), repeated."""
    import torch
    nbytes = 1 << 30
    x = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    ms = timed(lambda: x.mul_(1.0), max(5, args.steps), 2, torch.cuda.current_stream())
    print(json.dumps({"mode": "rmw", "bytes_read": nbytes, "bytes_written": nbytes,
                      "ms_per_pass": ms, "GBps": 2 * nbytes / (ms / 1e3) / 1e9}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--only", choices=["chunk", "decode"], default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--mode", choices=["bench", "copy", "rmw", "long", "gated", "bwd", "dec", "f32"],
                    default="bench")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported. The (batch, head) "
              "units are independent, so several GPUs would each run their own share.", file=sys.stderr)
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    from paper_2607_11897_amd import build, sfda
    if not os.path.exists(sfda.LIB_PATH):
        build.build(verbose=False)
    sfda.load_library()
    if args.mode == "copy":
        copy_calibration(args)
        return
    if args.mode == "rmw":
        rmw_calibration(args)
        return
    if args.mode == "long":
        long_context(args)
        return
    if args.mode == "gated":
        gated(args)
        return
    if args.mode == "bwd":
        backward(args)
        return
    if args.mode == "dec":
        decoupled(args)
        return
    if args.mode == "f32":
        fp32_forward(args)
        return
    stream = torch.cuda.current_stream()
    out = {}
    if args.only == "decode":
        out["decode"] = bench_decode(args, stream)
        print(json.dumps(out), flush=True)
        return
    if args.only is None:
        out["decode"] = bench_decode(args, stream)
    r = bench_chunk(args, stream)
    w = r["w"]
    line = {
        "metric": METRIC, "value": round(r["tokens_per_s"], 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(r["ms"], 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "H": w.H, "T": w.T, "d_k": 2 * w.m, "d_v": 2 * w.n,
                   "m_complex": w.m, "n_complex": w.n, "C": w.C, "state": "fp32", "accum": "fp32"},
        "launch_ms": r["launch_ms"],
        "launch_ms_c128": r["launch_ms_c128"],
        "roofline": r["roofline"],
    }
    if "decode" in out:
        line["decode"] = out["decode"]
    if not args.no_cpu_baseline:
        print("# timing the CPU oracle", file=sys.stderr, flush=True)
        line["cpu_baseline"] = cpu_baseline(r["x"])
    line["kernel_hash"] = kernel_hash()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
