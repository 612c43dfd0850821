"""Benchmark of the blockwise FP8 W8A8 linear-layer hot path on one MI355X.

One step = one pass of the whole path over one batch of synthetic input:
  1. weight re-quantisation   bf16 W [N][K] -> E4M3 + 128x128 fp32 block scales
  2. activation quantisation  bf16 A [M][K] -> E4M3 + 1x128 fp32 group scales
  3. blockwise FP8 GEMM       Y [M][N] bf16
on the Qwen3-8B-shaped prefill gate_up linear (M=8192 tokens, K=4096, N=24576),
with 1% outlier activation channels (x50) and 0.1% outlier weights (x20).

The JSON line's `value` is the step's effective GEMM throughput (2MNK per step
/ step time, TFLOP/s, all three kernels inside the timed region; 250 steps by
default, about 0.2 s, with the median and minimum of the per-step times beside
the mean).  `roofline` is the GEMM kernel alone, timed with HIP events on the
stream it runs on (mean, median and minimum launch).
`extra` carries the tiny configuration's step latency (64 x 512 x 512), the
same run's weight-resync figure (36 Qwen3-8B layers, 144
matrices, GB/s vs HBM), the MoE grouped GEMM (Qwen3-30B-A3B experts), the
decode linears of 36 distinct Qwen3-8B layers (M=256, weights from HBM), the
whole FP8 Qwen3-8B MLP (with the same MLP in bf16 through torch beside it) and
Qwen3-30B-A3B expert block, a plain device copy, and the rate of a register-fed
FP8 MFMA loop with its clock.
`cpu_baseline` times the CPU oracle on a bounded row sample of the same step.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
                       [--workload prefill|tiny|requant|moe|decode|mlp|moe_block|ue8m0|tis|kv|copy]
                       [--no-cpu-baseline] [--no-extra]
"""
import argparse
import json
import os
import sys
import time

import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import synth  # noqa: E402

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
FP8_PEAK_TFLOPS = 5000.0       # MI355X dense FP8 MFMA, TFLOP/s
METRIC = "blockwise FP8 GEMM TFLOP/s (% FP8 MFMA peak); weight requant GB/s (% HBM)"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=250)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="prefill", choices=["prefill", "tiny", "decode", "requant", "moe", "copy",
                                                              "mlp", "moe_block", "ue8m0", "tis", "kv", "dma", "loop"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra", action="store_true")
    ap.add_argument("--seed", type=int, default=3)
    return ap.parse_args()


class KernelTimer:
    """HIP events around individual launches on the current stream; averages per name."""

    def __init__(self):
        self.pending = []
        self.on = False

    def span(self, name):
        timer = self

        class _S:
            def __enter__(self):
                if timer.on:
                    self.e0 = torch.cuda.Event(enable_timing=True)
                    self.e1 = torch.cuda.Event(enable_timing=True)
                    self.e0.record()

            def __exit__(self, *a):
                if timer.on:
                    self.e1.record()
                    timer.pending.append((name, self.e0, self.e1))
        return _S()

    def samples_ms(self):
        torch.cuda.synchronize()
        acc = {}
        for name, e0, e1 in self.pending:
            acc.setdefault(name, []).append(e0.elapsed_time(e1))
        return acc

    def averages_ms(self):
        return {k: sum(v) / len(v) for k, v in self.samples_ms().items()}


def timed_loop(step, steps, warmup, timer, per_step=None):
    """Run `warmup` untimed steps, then time exactly `steps` steps between two events.
    Returns (mean ms per step, wall seconds); with per_step a list, each step's own
    event-timed duration (ms) is appended to it."""
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    timer.on = True
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)] if per_step is not None else None
    t0 = time.perf_counter()
    start.record()
    for i in range(steps):
        if marks:
            marks[i].record()
        step()
    if marks:
        marks[steps].record()
    stop.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    timer.on = False
    if marks:
        per_step.extend(marks[i].elapsed_time(marks[i + 1]) for i in range(steps))
    return start.elapsed_time(stop) / steps, wall


def median(xs):
    ys = sorted(xs)
    n = len(ys)
    return ys[n // 2] if n % 2 else 0.5 * (ys[n // 2 - 1] + ys[n // 2])


# ---------------------------------------------------------------------------
# prefill step (the headline workload)
# ---------------------------------------------------------------------------
def prefill(args, fp8rl):
    m, k, n = 8192, 4096, 24576
    a, w = synth.prefill_linear(seed=args.seed, device="cuda", m=m, k=k, n=n)
    qw = torch.empty((n, k), dtype=torch.uint8, device="cuda")
    sw = torch.empty((n // 128, k // 128), dtype=torch.float32, device="cuda")
    qa = torch.empty((m, k), dtype=torch.uint8, device="cuda")
    sa = torch.empty((k // 128, m), dtype=torch.float32, device="cuda")
    y = torch.empty((m, n), dtype=torch.bfloat16, device="cuda")
    timer = KernelTimer()

    def step():
        with timer.span("quant_weight"):
            fp8rl.fp8rl_quant_weight_block128(w, q=qw, scale=sw)
        with timer.span("quant_act"):
            fp8rl.fp8rl_quant_act_token_group128(a, q=qa, scale=sa)
        with timer.span("gemm"):
            fp8rl.fp8rl_gemm_w8a8_block(qa, sa, qw, sw, y=y)

    per_step = []
    ms, wall = timed_loop(step, args.steps, args.warmup, timer, per_step)
    samples = timer.samples_ms()
    kern = {kk: sum(v) / len(v) for kk, v in samples.items()}
    flops = 2.0 * m * n * k
    gemm_tflops = flops / (kern["gemm"] * 1e-3) / 1e12
    qw_bytes = n * k * 2 + n * k + (n // 128) * (k // 128) * 4
    qa_bytes = m * k * 2 + m * k + (k // 128) * m * 4
    prof = gemm_profile_figures()
    out = {
        "metric": METRIC,
        "value": round(flops / (ms * 1e-3) / 1e12, 2),
        "unit": "TFLOP/s",
        "ms_per_step": round(ms, 4),
        "ms_per_step_median": round(median(per_step), 4),
        "ms_per_step_min": round(min(per_step), 4),
        "wall_s_timed": round(wall, 3),
        "dtype": "fp8e4m3 x fp8e4m3 -> fp32 acc -> bf16",
        "config": {"workload": "Qwen3-8B prefill gate_up linear: weight requant + activation quant + "
                               "blockwise FP8 GEMM", "M": m, "K": k, "N": n,
                   "weight_block": [128, 128], "act_group": [1, 128], "seed": args.seed},
        "roofline": {
            "bound": "mfma", "achieved": round(gemm_tflops, 2), "peak": FP8_PEAK_TFLOPS,
            "unit": "TFLOP/s", "frac": round(gemm_tflops / FP8_PEAK_TFLOPS, 4), "traffic": prof["traffic"],
            "kernel": "gemm_w8a8_block", "avg_ms": round(kern["gemm"], 5),
            "median_ms": round(median(samples["gemm"]), 5), "min_ms": round(min(samples["gemm"]), 5),
            "launches_timed": len(samples["gemm"]),
            "algorithmic_flops_per_launch": flops,
            "traffic_unit": "bytes per launch crossing the L2-to-fabric boundary (rocprofv3 FETCH_SIZE + "
                            "WRITE_SIZE, calibrated on a device copy); the memory-side cache serves part of them",
            "sclk_GHz": prof["sclk_GHz"],
            "sclk_source": "GRBM_GUI_ACTIVE cycles per XCD over the dispatch duration, from the committed "
                           "counter profile of this kernel (null when the GEMM sources changed since)",
        },
        "kernels": {
            "quant_weight_block128": {"avg_ms": round(kern["quant_weight"], 5),
                                      "GB/s": round(qw_bytes / (kern["quant_weight"] * 1e-3) / 1e9, 1)},
            "quant_act_token_group128": {"avg_ms": round(kern["quant_act"], 5),
                                         "GB/s": round(qa_bytes / (kern["quant_act"] * 1e-3) / 1e9, 1)},
            "gemm_w8a8_block": {"avg_ms": round(kern["gemm"], 5), "TFLOP/s": round(gemm_tflops, 1)},
        },
    }
    return out, (a, w)


def prefill_ue8m0(args, fp8rl, steps=10, warmup=3):
    """The same prefill step with power-of-two (UE8M0) scales: both quantisers in
    their power-of-two form and the GEMM on the MX-scaled MFMA (section 2.4.3)."""
    m, k, n = 8192, 4096, 24576
    a, w = synth.prefill_linear(seed=args.seed, device="cuda", m=m, k=k, n=n)
    qw = torch.empty((n, k), dtype=torch.uint8, device="cuda")
    sw = torch.empty((n // 128, k // 128), dtype=torch.float32, device="cuda")
    qa = torch.empty((m, k), dtype=torch.uint8, device="cuda")
    sa = torch.empty((k // 128, m), dtype=torch.float32, device="cuda")
    y = torch.empty((m, n), dtype=torch.bfloat16, device="cuda")
    timer = KernelTimer()

    def step():
        with timer.span("quant_weight"):
            fp8rl.fp8rl_quant_weight_block128_ue8m0(w, q=qw, scale=sw)
        with timer.span("quant_act"):
            fp8rl.fp8rl_quant_act_token_group128_ue8m0(a, q=qa, scale=sa)
        with timer.span("gemm"):
            fp8rl.fp8rl_gemm_w8a8_block_ue8m0(qa, sa, qw, sw, y=y)

    ms, _ = timed_loop(step, steps, warmup, timer)
    kern = timer.averages_ms()
    flops = 2.0 * m * n * k
    t = flops / (kern["gemm"] * 1e-3) / 1e12
    res = {"workload": "Qwen3-8B prefill gate_up linear with power-of-two (UE8M0) scales: requant + quant + "
                       "GEMM on the MX-scaled MFMA", "ms_per_step": round(ms, 4),
           "kernels_ms": {kk: round(v, 5) for kk, v in kern.items()},
           "gemm_TFLOP/s": round(t, 1), "gemm_frac_fp8_peak": round(t / FP8_PEAK_TFLOPS, 4)}
    del a, w, qw, qa, y
    torch.cuda.empty_cache()
    return res


# ---------------------------------------------------------------------------
# the tiny configuration (64 x 512 x 512): latency of the whole step
# ---------------------------------------------------------------------------
def tiny(args, fp8rl, min_ms=250.0):
    """The whole step on the tiny linear (M=64, K=512, N=512): weight requant,
    activation quant and GEMM, three launches; steps are timed one by one over at
    least min_ms and reported as median and minimum (a latency, not a throughput)."""
    a, w = synth.tiny_linear(device="cuda")
    m, k = a.shape
    n = w.shape[0]
    qw = torch.empty((n, k), dtype=torch.uint8, device="cuda")
    sw = torch.empty((n // 128, k // 128), dtype=torch.float32, device="cuda")
    qa = torch.empty((m, k), dtype=torch.uint8, device="cuda")
    sa = torch.empty((k // 128, m), dtype=torch.float32, device="cuda")
    y = torch.empty((m, n), dtype=torch.bfloat16, device="cuda")

    def step():
        fp8rl.fp8rl_quant_weight_block128(w, q=qw, scale=sw)
        fp8rl.fp8rl_quant_act_token_group128(a, q=qa, scale=sa)
        fp8rl.fp8rl_gemm_w8a8_block(qa, sa, qw, sw, y=y)

    per_step = []
    total = 0.0
    while total < min_ms:
        ms, _ = timed_loop(step, 500, 20 if not per_step else 0, KernelTimer(), per_step)
        total += ms * 500
    # the same three launches replayed from a HIP graph: the GPU-side latency
    # without the host's per-launch cost
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        step()
        torch.cuda.synchronize()
        with torch.cuda.graph(graph, stream=side):
            step()
    torch.cuda.current_stream().wait_stream(side)
    per_replay = []
    total = 0.0
    while total < min_ms:
        ms, _ = timed_loop(graph.replay, 500, 20 if not per_replay else 0, KernelTimer(), per_replay)
        total += ms * 500
    del graph
    return {"workload": f"tiny blockwise W8A8 linear, M={m} K={k} N={n}: requant + quant + GEMM (3 launches)",
            "steps_timed": len(per_step), "us_per_step_median": round(median(per_step) * 1e3, 2),
            "us_per_step_min": round(min(per_step) * 1e3, 2),
            "graph_replays_timed": len(per_replay), "us_per_graph_replay_median": round(median(per_replay) * 1e3, 2),
            "us_per_graph_replay_min": round(min(per_replay) * 1e3, 2),
            "GEMM_MFLOP": 2.0 * m * n * k / 1e6}


# ---------------------------------------------------------------------------
# weight resync: 36 layers x 4 matrices
# ---------------------------------------------------------------------------
def requant(args, fp8rl, steps=5, warmup=2):
    """All 144 weight matrices of 36 Qwen3-8B layers, each re-quantised once per
    pass (20.8 GB of HBM traffic, far beyond the 256 MB last-level cache, so every
    pass is cold).  The pass is one fp8rl_quant_weight_block128_batched call (three
    launches of at most 64 matrices); the same pass as 144 single-matrix launches
    is timed beside it.  Each is captured in a HIP graph, as a weight-sync loop
    would issue it, and the graph is replayed."""
    mats = []
    for layer in range(synth.QWEN3_8B_LAYERS):
        for name in synth.QWEN3_8B_LINEARS:
            w, _, _ = synth.requant_matrix(layer, name, device="cuda")
            n, k = w.shape
            mats.append((w, torch.empty((n, k), dtype=torch.uint8, device="cuda"),
                         torch.empty((n // 128, k // 128), dtype=torch.float32, device="cuda")))
    elems = sum(w.numel() for w, _, _ in mats)
    nbytes = sum(w.numel() * 3 + s.numel() * 4 for w, _, s in mats)
    ws, qs, ss = zip(*mats)

    def batched_pass():
        fp8rl.fp8rl_quant_weight_block128_batched(ws, qs, ss)

    def per_matrix_pass():
        for w, q, s in mats:
            fp8rl.fp8rl_quant_weight_block128(w, q=q, scale=s)

    def time_graph(one_pass):
        one_pass()                               # eager warm-up (also loads the kernel)
        torch.cuda.synchronize()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.stream(side):
            with torch.cuda.graph(graph, stream=side):
                one_pass()
        torch.cuda.current_stream().wait_stream(side)
        for _ in range(warmup):
            graph.replay()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            graph.replay()
        e1.record()
        torch.cuda.synchronize()
        del graph
        return e0.elapsed_time(e1) / steps

    ms = time_graph(batched_pass)
    ms_single = time_graph(per_matrix_pass)
    gbs = nbytes / (ms * 1e-3) / 1e9
    gbs_single = nbytes / (ms_single * 1e-3) / 1e9
    del mats, ws, qs, ss
    torch.cuda.empty_cache()
    return {"workload": "weight resync, 36 Qwen3-8B layers x {qkv, o_proj, gate_up, down}: one batched call "
                        "(3 launches) replayed from a HIP graph",
            "elements": elems, "bytes": nbytes, "ms_per_pass": round(ms, 4),
            "GB/s": round(gbs, 1), "frac_hbm": round(gbs / HBM_PEAK_GBS, 4),
            "per_matrix_launches": {"ms_per_pass": round(ms_single, 4), "GB/s": round(gbs_single, 1),
                                    "frac_hbm": round(gbs_single / HBM_PEAK_GBS, 4)}}


def hbm_copy_reference(nbytes=4 << 30, steps=5):
    """Plain device-to-device copy of a buffer 16x the last-level cache: the
    practical read+write HBM rate of this GPU, for context next to the spec."""
    src = torch.empty(nbytes // 2, dtype=torch.bfloat16, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    del src, dst
    torch.cuda.empty_cache()
    return round(2 * nbytes / (ms * 1e-3) / 1e9, 1)


def dma_probe(args, fp8rl, region_kib=(16, 64, 256, 2048), waves=(4, 8, 16), inflight=(2, 8)):
    """Rate of the global-to-LDS DMA alone (libfp8rl_probe.so), and of the same
    16-byte loads into registers, one workgroup per CU, each streaming its own
    region: regions of 16 KiB stay in the CU's L1, of 64 KiB (16 MiB over all
    CUs) in the L2s, of 256 KiB in the memory-side cache, of 2 MiB (512 MiB) in
    HBM.  Per CU: bytes per shader clock."""
    import ctypes
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2601_18150_amd", "libfp8rl_probe.so"))
    fn = lib.fp8rl_probe_dma_rate
    fn.argtypes = [ctypes.c_void_p, ctypes.c_longlong, ctypes.c_longlong, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                   ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    blocks = torch.cuda.get_device_properties(0).multi_processor_count
    src_bytes = blocks * max(region_kib) * 1024
    src = torch.ones(src_bytes, dtype=torch.uint8, device="cuda")
    sink = torch.empty(blocks * 16 * 64, dtype=torch.float32, device="cuda")
    clk = torch.zeros(2 * blocks, dtype=torch.int64, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    rows = []
    for to_lds, rk, w, n in ((d, r, w, n) for d in (1, 0) for r in region_kib for w in waves for n in inflight):
        per_iter = blocks * w * n * 1024
        iters = max(4, (1 << 30) // per_iter)           # about 1 GiB per run
        call = (src.data_ptr(), src_bytes, rk * 1024, blocks, w, n, to_lds, iters, sink.data_ptr(),
                clk.data_ptr(), stream)
        if fn(*call) != 0:
            raise RuntimeError("DMA probe launch failed")
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        fn(*call)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        c = clk.view(blocks, 2).double()
        ghz = (c[:, 0].sum() / c[:, 1].sum()).item() * 0.1
        moved = per_iter * iters
        rows.append({"into": "LDS" if to_lds else "registers", "region_KiB": rk, "waves": w, "inflight": n,
                     "TB/s": round(moved / (ms * 1e-3) / 1e12, 3),
                     "B_per_clk_per_CU": round(moved / blocks / (ms * 1e-3 * ghz * 1e9), 2),
                     "clock_GHz": round(ghz, 3)})
    del src, sink
    torch.cuda.empty_cache()
    return {"workload": f"global-to-LDS DMA and register loads alone, {blocks} workgroups (one per CU), 16 bytes "
                        f"per lane",
            "rows": rows}


def mfma_loop_probe(args, fp8rl, iters=4000):
    """The GEMM K step's inner loop without memory traffic (libfp8rl_probe.so):
    fragment reads from LDS and MFMAs on the prefill's 128n x 64m and the decode /
    MoE 64n x 64m wave tiles, 8 waves per CU, with and without the per-K-block
    scale FMAs and the per-step barrier; TFLOP/s against the spec peak and the
    register-fed MFMA loop of the same run (which holds a lower clock)."""
    import ctypes
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2601_18150_amd", "libfp8rl_probe.so"))
    fn = lib.fp8rl_probe_mfma_loop
    fn.argtypes = [ctypes.c_int] * 5 + [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    blocks = torch.cuda.get_device_properties(0).multi_processor_count
    out = torch.empty(blocks * 512, dtype=torch.float32, device="cuda")
    clk = torch.zeros(2 * blocks, dtype=torch.int64, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    ref = mfma_probe()
    rows = []
    for tile, (tn, tm) in ((0, (8, 4)), (1, (4, 4))):
        for fma in (0, 1):
            for barrier in (0, 1):
                call = (tile, fma, barrier, blocks, iters, out.data_ptr(), clk.data_ptr(), stream)
                if fn(*call) != 0:
                    raise RuntimeError("inner-loop probe launch failed")
                torch.cuda.synchronize()
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record()
                fn(*call)
                e1.record()
                torch.cuda.synchronize()
                ms = e0.elapsed_time(e1)
                c = clk.view(blocks, 2).double()
                ghz = (c[:, 0].sum() / c[:, 1].sum()).item() * 0.1
                flops = blocks * 8 * iters * tn * tm * 2.0 * 16 * 16 * 128
                tf = flops / (ms * 1e-3) / 1e12
                rows.append({"wave_tile": f"{16 * tn}n x {16 * tm}m", "scale_fma": bool(fma), "barrier": bool(barrier),
                             "TFLOP/s": round(tf, 1), "frac_of_spec": round(tf / FP8_PEAK_TFLOPS, 4),
                             "frac_of_mfma_loop": round(tf / ref["TFLOP/s"], 4), "clock_GHz": round(ghz, 3)})
    return {"workload": f"GEMM K-step inner loop alone: LDS fragment reads + MFMAs, {blocks} workgroups of 8 waves",
            "mfma_loop_reference": ref, "rows": rows}


# ---------------------------------------------------------------------------
# MoE grouped GEMM (gate_up and down)
# ---------------------------------------------------------------------------
def moe(args, fp8rl, steps=10, warmup=3):
    lay = synth.moe_layer(device="cuda")
    off = lay["routing"].offsets.to("cuda")
    counts = lay["routing"].counts
    res = {}
    for which in ("gate_up", "down"):
        x = lay["x_gate_up"] if which == "gate_up" else lay["x_down"]
        wts = lay["w_gate_up"] if which == "gate_up" else lay["w_down"]
        g, n, k = wts.shape
        qw, sw = fp8rl.fp8rl_quant_weight_block128(wts.reshape(g * n, k))
        qw = qw.reshape(g, n, k)
        sw = sw.reshape(g, n // 128, k // 128)
        qa, sa = fp8rl.fp8rl_quant_act_token_group128(x)
        y = torch.empty((x.shape[0], n), dtype=torch.bfloat16, device="cuda")
        timer = KernelTimer()

        def step():
            with timer.span("grouped"):
                fp8rl.fp8rl_grouped_gemm_w8a8_block(qa, sa, qw, sw, off, y=y)

        timed_loop(step, steps, warmup, timer)
        kms = timer.averages_ms()["grouped"]
        rows = x.shape[0]
        flops = 2.0 * rows * n * k
        active = int((counts > 0).sum())
        nbytes = active * n * k + rows * k + rows * n * 2 + rows * (k // 128) * 4
        t = flops / (kms * 1e-3) / 1e12
        roof_ms = max(flops / (FP8_PEAK_TFLOPS * 1e12), nbytes / (HBM_PEAK_GBS * 1e9)) * 1e3
        res[which] = {"N": n, "K": k, "rows": rows, "active_experts": active, "avg_ms": round(kms, 5),
                      "TFLOP/s": round(t, 1), "frac_fp8_peak": round(t / FP8_PEAK_TFLOPS, 4),
                      "GB/s_min_traffic": round(nbytes / (kms * 1e-3) / 1e9, 1),
                      "min_traffic_bytes": nbytes, "roofline_ms": round(roof_ms, 5),
                      "frac_min_roofline": round(roof_ms / kms, 4)}
    del lay
    torch.cuda.empty_cache()
    return res


# ---------------------------------------------------------------------------
# whole FP8 MLP blocks: dense Qwen3-8B MLP and one Qwen3-30B-A3B MoE expert block
# ---------------------------------------------------------------------------
def _silu_quant_bytes(m, inter):
    """Algorithmic HBM bytes of the fused SiLU*mul + quantisation (h not written):
    read gate and up (bf16), write codes and one fp32 scale per 128 elements."""
    return m * inter * 4 + m * inter + m * (inter // 128) * 4


def mlp(args, fp8rl, steps=10, warmup=3):
    """Qwen3-8B MLP forward at prefill (8192 tokens): quantise x, gate_up GEMM
    (N=24576), fused SiLU*mul + 1x128 quantisation, down GEMM (K=12288), all in
    FP8 with the weights pre-quantised; next to it the same MLP in bf16 through
    torch (hipBLASLt GEMMs, SiLU and product as separate elementwise kernels)."""
    m, h, inter = 8192, 4096, 12288
    x = synth.normal_bf16((m, h), 1.0, 50, "cuda")
    w_gu = synth.normal_bf16((2 * inter, h), 0.02, 51, "cuda")
    w_dn = synth.normal_bf16((h, inter), 0.02, 52, "cuda")
    qgu, sgu = fp8rl.fp8rl_quant_weight_block128(w_gu)
    qdn, sdn = fp8rl.fp8rl_quant_weight_block128(w_dn)
    qx = torch.empty((m, h), dtype=torch.uint8, device="cuda")
    sx = torch.empty((h // 128, m), dtype=torch.float32, device="cuda")
    gu = torch.empty((m, 2 * inter), dtype=torch.bfloat16, device="cuda")
    qh = torch.empty((m, inter), dtype=torch.uint8, device="cuda")
    sh = torch.empty((inter // 128, m), dtype=torch.float32, device="cuda")
    y = torch.empty((m, h), dtype=torch.bfloat16, device="cuda")
    timer = KernelTimer()

    def step():
        with timer.span("quant_act"):
            fp8rl.fp8rl_quant_act_token_group128(x, q=qx, scale=sx)
        with timer.span("gemm_gate_up"):
            fp8rl.fp8rl_gemm_w8a8_block(qx, sx, qgu, sgu, y=gu)
        with timer.span("silu_mul_quant"):
            fp8rl.fp8rl_silu_mul_quant_group128(gu, q=qh, scale=sh)
        with timer.span("gemm_down"):
            fp8rl.fp8rl_gemm_w8a8_block(qh, sh, qdn, sdn, y=y)

    ms, _ = timed_loop(step, steps, warmup, timer)
    kern = timer.averages_ms()
    wt_gu, wt_dn = w_gu.t().contiguous(), w_dn.t().contiguous()

    def step_bf16():
        g = torch.matmul(x, wt_gu)
        hh = torch.nn.functional.silu(g[:, :inter]) * g[:, inter:]
        torch.matmul(hh, wt_dn)

    ms_bf16, _ = timed_loop(step_bf16, steps, warmup, KernelTimer())
    flops = 2.0 * m * h * 2 * inter + 2.0 * m * inter * h
    sq = _silu_quant_bytes(m, inter)
    res = {"workload": f"Qwen3-8B MLP forward, {m} tokens: quant x, gate_up GEMM, fused SiLU*mul+quant, "
                       f"down GEMM (weights pre-quantised)",
           "ms_per_step": round(ms, 4), "TFLOP/s": round(flops / (ms * 1e-3) / 1e12, 1),
           "bf16_torch_ms_per_step": round(ms_bf16, 4), "speedup_vs_bf16_torch": round(ms_bf16 / ms, 3),
           "kernels_ms": {k: round(v, 5) for k, v in kern.items()},
           "silu_mul_quant": {"bytes": sq, "GB/s": round(sq / (kern["silu_mul_quant"] * 1e-3) / 1e9, 1),
                              "frac_hbm": round(sq / (kern["silu_mul_quant"] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}}
    del x, w_gu, w_dn, qgu, qdn, gu, qh, y, wt_gu, wt_dn
    torch.cuda.empty_cache()
    return res


def moe_block(args, fp8rl, steps=10, warmup=3):
    """One Qwen3-30B-A3B expert block (4096 tokens, top-8 of 128 experts, hidden
    2048, expert intermediate 768) end to end in FP8: quantise the tokens once,
    grouped gate_up GEMM reading the routed token rows in expert order, fused
    SiLU*mul + quantisation, grouped down GEMM; beside it the same block with the
    dispatch as a separate gather of the quantised rows."""
    lay = synth.moe_layer(device="cuda")
    routing = lay["routing"]
    off = routing.offsets.to("cuda")
    idx = routing.token_of_row.to(torch.int32).to("cuda")
    tokens, hidden = 4096, lay["w_gate_up"].shape[2]
    x_tok = synth.normal_bf16((tokens, hidden), 1.0, 6 + 11, "cuda")
    qw = {}
    for which in ("w_gate_up", "w_down"):
        g, n, k = lay[which].shape
        q, s = fp8rl.fp8rl_quant_weight_block128(lay[which].reshape(g * n, k))
        qw[which] = (q.reshape(g, n, k), s.reshape(g, n // 128, k // 128))
    inter = lay["w_down"].shape[2]
    rows = idx.numel()
    del lay
    torch.cuda.empty_cache()
    qx = torch.empty((tokens, hidden), dtype=torch.uint8, device="cuda")
    sx = torch.empty((hidden // 128, tokens), dtype=torch.float32, device="cuda")
    qr = torch.empty((rows, hidden), dtype=torch.uint8, device="cuda")
    sr = torch.empty((hidden // 128, rows), dtype=torch.float32, device="cuda")
    gu = torch.empty((rows, 2 * inter), dtype=torch.bfloat16, device="cuda")
    qh = torch.empty((rows, inter), dtype=torch.uint8, device="cuda")
    sh = torch.empty((inter // 128, rows), dtype=torch.float32, device="cuda")
    y = torch.empty((rows, hidden), dtype=torch.bfloat16, device="cuda")
    timer = KernelTimer()

    def step():
        # dispatch fused into the gate_up GEMM: it reads each expert row's token
        # codes and scales through the routing index
        with timer.span("quant_act"):
            fp8rl.fp8rl_quant_act_token_group128(x_tok, q=qx, scale=sx)
        with timer.span("grouped_gate_up_gathered"):
            fp8rl.fp8rl_grouped_gemm_w8a8_block_gathered(qx, sx, idx, *qw["w_gate_up"], off, y=gu)
        with timer.span("silu_mul_quant"):
            fp8rl.fp8rl_silu_mul_quant_group128(gu, q=qh, scale=sh)
        with timer.span("grouped_down"):
            fp8rl.fp8rl_grouped_gemm_w8a8_block(qh, sh, *qw["w_down"], off, y=y)

    def step_copy():
        # the same block with the dispatch as a separate gather of quantised rows
        with timer.span("c_quant_act"):
            fp8rl.fp8rl_quant_act_token_group128(x_tok, q=qx, scale=sx)
        with timer.span("c_gather_rows"):
            fp8rl.fp8rl_gather_rows_fp8(qx, sx, idx, q_dst=qr, s_dst=sr)
        with timer.span("c_grouped_gate_up"):
            fp8rl.fp8rl_grouped_gemm_w8a8_block(qr, sr, *qw["w_gate_up"], off, y=gu)
        with timer.span("c_silu_mul_quant"):
            fp8rl.fp8rl_silu_mul_quant_group128(gu, q=qh, scale=sh)
        with timer.span("c_grouped_down"):
            fp8rl.fp8rl_grouped_gemm_w8a8_block(qh, sh, *qw["w_down"], off, y=y)

    ms, _ = timed_loop(step, steps, warmup, timer)
    ms_copy, _ = timed_loop(step_copy, steps, warmup, timer)
    kern = timer.averages_ms()
    flops = 2.0 * rows * hidden * 2 * inter + 2.0 * rows * inter * hidden
    sq = _silu_quant_bytes(rows, inter)
    gb = 2 * rows * hidden + 2 * rows * (hidden // 128) * 4
    res = {"workload": f"Qwen3-30B-A3B expert block, {tokens} tokens x top-8 -> {rows} rows: quant, grouped "
                       f"gate_up over the routed token rows, fused SiLU*mul+quant, grouped down",
           "ms_per_step": round(ms, 4), "TFLOP/s": round(flops / (ms * 1e-3) / 1e12, 1),
           "kernels_ms": {k: round(v, 5) for k, v in kern.items() if not k.startswith("c_")},
           "silu_mul_quant": {"bytes": sq, "GB/s": round(sq / (kern["silu_mul_quant"] * 1e-3) / 1e9, 1)},
           "with_separate_gather": {"ms_per_step": round(ms_copy, 4),
                                    "kernels_ms": {k[2:]: round(v, 5) for k, v in kern.items() if k.startswith("c_")},
                                    "gather_rows": {"bytes": gb, "GB/s": round(gb / (kern["c_gather_rows"] * 1e-3)
                                                                              / 1e9, 1)}}}
    del qw, x_tok, qx, qr, gu, qh, y
    torch.cuda.empty_cache()
    return res


def tis_step(args, fp8rl, steps=20, warmup=5):
    """Token-level TIS weights and mismatch-KL sums over one rollout batch (32 prompts x
    16 samples x 20480 tokens, padding masked), C = 2: HIP events around each call,
    and 20 calls back to back replayed from a HIP graph."""
    lt, lr, mask = synth.rollout_logprobs(device="cuda")
    n = lt.numel()
    w = torch.empty(n, dtype=torch.float32, device="cuda")
    stats = torch.empty(4, dtype=torch.float64, device="cuda")
    work = torch.empty(fp8rl.fp8rl_tis_workspace_size(n), dtype=torch.uint8, device="cuda")
    timer = KernelTimer()

    def step():
        with timer.span("tis"):
            fp8rl.fp8rl_tis_weights_kl(lt, lr, mask, 2.0, w_tis=w, stats=stats, workspace=work)

    timed_loop(step, steps, warmup, timer)
    ms = timer.averages_ms()["tis"]
    # the same call 20 times back to back in a HIP graph: per-call time without the
    # launch and event overhead that dominates a single 25 us call's span
    calls = 20
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        fp8rl.fp8rl_tis_weights_kl(lt, lr, mask, 2.0, w_tis=w, stats=stats, workspace=work)
        torch.cuda.synchronize()
        with torch.cuda.graph(graph, stream=side):
            for _ in range(calls):
                fp8rl.fp8rl_tis_weights_kl(lt, lr, mask, 2.0, w_tis=w, stats=stats, workspace=work)
    torch.cuda.current_stream().wait_stream(side)
    graph_ms, _ = timed_loop(graph.replay, 10, 2, KernelTimer())
    del graph
    per_call = graph_ms / calls
    nbytes = n * (4 + 4 + 1 + 4)
    res = {"workload": f"TIS weights + mismatch-KL sums, {n} rollout tokens (32 x 16 x 20480)",
           "avg_ms": round(ms, 5), "bytes": nbytes, "GB/s": round(nbytes / (ms * 1e-3) / 1e9, 1),
           "frac_hbm": round(nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
           "graph_ms_per_call": round(per_call, 5),
           "graph_GB/s": round(nbytes / (per_call * 1e-3) / 1e9, 1),
           "graph_frac_hbm": round(nbytes / (per_call * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
    del lt, lr, mask, w, work
    torch.cuda.empty_cache()
    return res


def kv_decode(args, fp8rl, steps=10, warmup=3):
    """One Qwen3-8B attention layer at decode (32 query heads, 8 kv heads of 128) over a
    paged cache: 64 sequences of 4096 .. 20480 tokens (seeded), the FP8 cache against the
    same kernel over a bf16 cache, plus the per-step calibration and the cache write."""
    g = torch.Generator(device="cpu")
    g.manual_seed(11)
    batch, qh, kvh = 64, 32, 8
    seq = torch.randint(4096, 20481, (batch,), generator=g, dtype=torch.int32)
    pages = (seq + 15) // 16
    nb = int(pages.sum())
    perm = torch.randperm(nb, generator=g).to(torch.int32)
    max_blocks = int(pages.max())
    table = torch.zeros((batch, max_blocks), dtype=torch.int32)
    off = 0
    for b in range(batch):
        table[b, :pages[b]] = perm[off:off + int(pages[b])]
        off += int(pages[b])
    table, seq_d = table.cuda(), seq.cuda()
    max_seq = int(seq.max())
    dev = torch.Generator(device="cuda")
    dev.manual_seed(12)
    # keys and values: N(0,1) bf16 (written page by page through the FP8 write kernel below)
    kb = torch.randn((nb, kvh, 16, 128), generator=dev, device="cuda").to(torch.bfloat16)
    vb = torch.randn((nb, kvh, 4, 128, 4), generator=dev, device="cuda").to(torch.bfloat16)   # value page layout
    q = torch.randn((batch, qh, 128), generator=dev, device="cuda").to(torch.bfloat16)
    ks = fp8rl.fp8rl_kv_calibrate_scale(kb)
    vs = fp8rl.fp8rl_kv_calibrate_scale(vb)
    kc = torch.empty((nb, kvh, 16, 128), dtype=torch.uint8, device="cuda")
    vc = torch.empty((nb, kvh, 4, 128, 4), dtype=torch.uint8, device="cuda")
    # every cache slot once, in slot order (slot = block * 16 + 4a + c)
    tok_k = kb.permute(0, 2, 1, 3).reshape(nb * 16, kvh, 128).contiguous()
    tok_v = vb.permute(0, 2, 4, 1, 3).reshape(nb * 16, kvh, 128).contiguous()
    slots = torch.arange(nb * 16, dtype=torch.int64, device="cuda")
    timer = KernelTimer()
    sm = 1.0 / 128 ** 0.5
    work = torch.empty(fp8rl.fp8rl_attention_decode_workspace_size(batch, qh, kvh, max_seq), dtype=torch.uint8,
                       device="cuda")
    out = torch.empty_like(q)

    def step():
        with timer.span("calibrate_k"):
            fp8rl.fp8rl_kv_calibrate_scale(tok_k, scale=ks)
        with timer.span("cache_write"):
            fp8rl.fp8rl_kv_cache_write_fp8(tok_k, tok_v, slots, ks, vs, kc, vc)
        with timer.span("attn_fp8"):
            fp8rl.fp8rl_attention_decode_fp8kv(q, kc, vc, table, seq_d, max_seq, ks, vs, sm, out=out, workspace=work)
        with timer.span("attn_bf16"):
            fp8rl.fp8rl_attention_decode_bf16kv(q, kb, vb, table, seq_d, max_seq, sm, out=out, workspace=work)

    timed_loop(step, steps, warmup, timer)
    kern = timer.averages_ms()
    tokens = int(seq.sum())
    cache_fp8 = tokens * kvh * 128 * 2
    write_bytes = nb * 16 * kvh * 128 * (2 + 2 + 1 + 1)      # bf16 K and V in, their codes out (every slot)
    calib_bytes = nb * 16 * kvh * 128 * 2                    # bf16 keys read
    res = {"workload": f"Qwen3-8B decode attention layer, {batch} sequences of 4096..20480 tokens ({tokens} cached "
                       f"tokens), paged FP8 cache vs bf16 cache",
           "kernels_ms": {k: round(v, 5) for k, v in kern.items()},
           "attn_fp8": {"bytes": cache_fp8, "GB/s": round(cache_fp8 / (kern["attn_fp8"] * 1e-3) / 1e9, 1),
                        "frac_hbm": round(cache_fp8 / (kern["attn_fp8"] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)},
           "attn_bf16": {"bytes": 2 * cache_fp8, "GB/s": round(2 * cache_fp8 / (kern["attn_bf16"] * 1e-3) / 1e9, 1)},
           "cache_write": {"tokens": nb * 16, "bytes": write_bytes,
                           "GB/s": round(write_bytes / (kern["cache_write"] * 1e-3) / 1e9, 1),
                           "frac_hbm": round(write_bytes / (kern["cache_write"] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)},
           "calibrate_k": {"bytes": calib_bytes, "GB/s": round(calib_bytes / (kern["calibrate_k"] * 1e-3) / 1e9, 1),
                           "frac_hbm": round(calib_bytes / (kern["calibrate_k"] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)},
           "fp8_speedup_vs_bf16_cache": round(kern["attn_bf16"] / kern["attn_fp8"], 3)}
    del kb, vb, kc, vc, tok_k, tok_v, work
    torch.cuda.empty_cache()
    return res


# ---------------------------------------------------------------------------
# decode linears of one Qwen3-8B layer (M=256): GEMM timing per linear
# ---------------------------------------------------------------------------
def decode(args, fp8rl, sweeps=3, warmup=1, layers=synth.QWEN3_8B_LAYERS):
    """The four decode linears (M=256) of 36 distinct Qwen3-8B layers, 144 GEMMs per
    sweep: the 6.95 GB of weight codes exceed the last-level cache, so every layer's
    weights come from HBM as in a real decode step."""
    acts = synth.decode_activations(device="cuda")
    q_in = {kin: fp8rl.fp8rl_quant_act_token_group128(acts["h" if kin == 4096 else "inter"])
            for kin in (4096, 12288)}
    m = acts["h"].shape[0]
    del acts
    qws = []
    for layer in range(layers):
        wts = synth.layer_weights(layer, device="cuda")
        qws.append({name: fp8rl.fp8rl_quant_weight_block128(w) for name, w in wts.items()})
        del wts
    torch.cuda.empty_cache()
    ys = {name: torch.empty((m, n), dtype=torch.bfloat16, device="cuda")
          for name, (k, n) in synth.QWEN3_8B_LINEARS.items()}
    # split-K workspace: one buffer, large enough for every linear (calls are stream-ordered)
    ws_bytes = max(fp8rl.fp8rl_gemm_w8a8_block_workspace_size(m, n, k)
                   for k, n in synth.QWEN3_8B_LINEARS.values())
    work = torch.empty(max(ws_bytes, 16), dtype=torch.uint8, device="cuda")
    timer = KernelTimer()

    def sweep():
        for layer in range(layers):
            for name, (k, n) in synth.QWEN3_8B_LINEARS.items():
                qa, sa = q_in[k]
                qw, sw = qws[layer][name]
                with timer.span(name):
                    fp8rl.fp8rl_gemm_w8a8_block_ws(qa, sa, qw, sw, work, y=ys[name])

    # per-GEMM durations from an eager sweep (HIP events around each launch) ...
    timed_loop(sweep, 1, warmup, timer)
    avg = timer.averages_ms()
    # ... and the sweep itself replayed from one HIP graph, so that host-side launch
    # cost (144 launches through the Python binding) does not open gaps between kernels
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side):
        sweep()                                   # warm-up on the capture stream
        torch.cuda.synchronize()
        with torch.cuda.graph(graph, stream=side):
            sweep()
    torch.cuda.current_stream().wait_stream(side)
    graph.replay()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(sweeps):
        graph.replay()
    e1.record()
    torch.cuda.synchronize()
    sweep_ms = e0.elapsed_time(e1) / sweeps
    del graph
    flops = bytes_ = 0.0
    res = {"workload": f"decode linears of {layers} distinct Qwen3-8B layers (M={m}), "
                       f"{4 * layers} GEMMs per sweep, weights from HBM, split-K workspace {ws_bytes} bytes"}
    for name, (k, n) in synth.QWEN3_8B_LINEARS.items():
        f = 2.0 * m * n * k
        nb = n * k + m * k + m * n * 2 + (n // 128) * (k // 128) * 4 + m * (k // 128) * 4
        flops += f * layers
        bytes_ += nb * layers
        res[name] = {"K": k, "N": n, "avg_ms": round(avg[name], 5),
                     "TFLOP/s": round(f / (avg[name] * 1e-3) / 1e12, 1),
                     "GB/s_min_traffic": round(nb / (avg[name] * 1e-3) / 1e9, 1)}
    roof_ms = max(flops / (FP8_PEAK_TFLOPS * 1e12), bytes_ / (HBM_PEAK_GBS * 1e9)) * 1e3
    res.update({"sweep_ms": round(sweep_ms, 4), "TFLOP/s": round(flops / (sweep_ms * 1e-3) / 1e12, 1),
                "GB/s_min_traffic": round(bytes_ / (sweep_ms * 1e-3) / 1e9, 1),
                "roofline_ms": round(roof_ms, 4), "frac_roofline": round(roof_ms / sweep_ms, 4)})
    del qws, ys, q_in
    torch.cuda.empty_cache()
    return res


def mfma_probe(blocks_per_cu=2, iters=20000):
    """Measured FP8 MFMA rate of a register-fed MFMA loop (libfp8rl_probe.so) and
    the shader clock it ran at (s_memtime ticks per 100 MHz real-time tick)."""
    import ctypes
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2601_18150_amd", "libfp8rl_probe.so"))
    fn = lib.fp8rl_probe_mfma_rate
    fn.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p]
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    blocks = cus * blocks_per_cu
    out = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")
    clk = torch.zeros(2 * blocks, dtype=torch.int64, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    best = None
    for _ in range(3):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        if fn(out.data_ptr(), clk.data_ptr(), blocks, iters, stream) != 0:
            raise RuntimeError("MFMA probe launch failed")
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        if best is None or ms < best[0]:
            c = clk.view(blocks, 2).double()
            best = (ms, (c[:, 0].sum() / c[:, 1].sum()).item() * 0.1)
    ms, ghz = best
    flops = blocks * 4 * iters * 4 * 2.0 * 16 * 16 * 128
    t = flops / (ms * 1e-3) / 1e12
    return {"TFLOP/s": round(t, 1), "frac_of_spec": round(t / FP8_PEAK_TFLOPS, 4), "clock_GHz": round(ghz, 3),
            "what": "register-fed 16x16x128 FP8 MFMA loop, 2 waves per SIMD"}


# ---------------------------------------------------------------------------
# CPU oracle baseline on a bounded sample of the prefill step
# ---------------------------------------------------------------------------
GEMM_SOURCES = ["gemm_core.hpp", "gemm.hip", "common.hpp"]
TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "gemm_prefill_gate_up_traffic.md")
COUNTERS_PROFILE = os.path.join(ROOT, "profiles", "gemm_prefill_gate_up_counters.md")


def _profile_fields(path, keys):
    """key: value lines of a committed profile summary, or None when the GEMM
    sources changed since it was taken (its source_sha256 line no longer matches)."""
    import hashlib
    try:
        text = open(path).read()
    except OSError:
        return None
    h = hashlib.sha256()
    for f in GEMM_SOURCES:
        with open(os.path.join(ROOT, "paper_2601_18150_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    fields = dict(ln.split(":", 1) for ln in text.splitlines() if ln.startswith(tuple(k + ":" for k in keys)))
    if fields.get("source_sha256", "").strip() != h.hexdigest()[:16]:
        return None
    return {k: v.strip() for k, v in fields.items()}


def gemm_profile_figures():
    """HBM-side bytes per GEMM launch (rocprofv3 FETCH_SIZE / WRITE_SIZE, calibrated on
    a device copy) and the engine clock during the GEMM (GRBM_GUI_ACTIVE), each read
    from its committed profile summary; None where the GEMM sources changed since."""
    tr = _profile_fields(TRAFFIC_PROFILE, ("hbm_bytes_per_launch", "source_sha256"))
    ck = _profile_fields(COUNTERS_PROFILE, ("sclk_GHz", "source_sha256"))
    return {"traffic": int(tr["hbm_bytes_per_launch"]) if tr and "hbm_bytes_per_launch" in tr else None,
            "sclk_GHz": float(ck["sclk_GHz"]) if ck and "sclk_GHz" in ck else None}


def cpu_baseline(a, w, chunk=1024, min_seconds=10.0):
    """The numpy oracle on the host, as a reported baseline: quantise all weights,
    then quantise and multiply 1024-row chunks of the activations until
    min_seconds have passed or all rows are done (the sample is stated)."""
    import numpy as np
    from oracle import gemm, quant
    cores = len(os.sched_getaffinity(0))
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        blas_threads = None
    m, k = a.shape
    n = w.shape[0]
    w_h = w.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    a_h = a.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    t0 = time.perf_counter()
    qw, sw = quant.quant_weight_block128(w_h)
    rows = 0
    while rows < m and (rows == 0 or time.perf_counter() - t0 < min_seconds):
        r1 = min(rows + chunk, m)
        qa, sa = quant.quant_act_token_group128(a_h[rows:r1])
        gemm.gemm_ref_fp64(qa, sa, qw, sw)
        rows = r1
    dt = time.perf_counter() - t0
    flops = 2.0 * rows * n * k
    return {"value": round(flops / dt / 1e12, 6), "unit": "TFLOP/s", "cores": cores, "blas_threads": blas_threads,
            "kind": "oracle",
            "sample": f"first {rows} of {m} token rows through the full step (weight quantisation of all "
                      f"{n}x{k} weights once, activation quantisation, fp64 GEMM in {chunk}-row chunks until "
                      f"{min_seconds:.0f} s had passed); {dt:.1f} s on the host",
            "seconds": round(dt, 2)}


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "bench.py runs on one GPU; runs on several GPUs are not supported",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    import paper_2601_18150_amd as fp8rl
    fp8rl.load()
    torch.cuda.init()
    if args.workload != "prefill":
        if args.workload == "copy":
            print(json.dumps({"workload": "device-to-device copy of 4 GiB (torch copy_)",
                              "GB/s": hbm_copy_reference()}), flush=True)
            return
        fn = {"tiny": tiny, "requant": requant, "moe": moe, "decode": decode, "mlp": mlp, "moe_block": moe_block,
              "ue8m0": prefill_ue8m0, "tis": tis_step, "kv": kv_decode, "dma": dma_probe, "loop": mfma_loop_probe}[args.workload]
        print(json.dumps(fn(args, fp8rl)), flush=True)
        return
    out, (a, w) = prefill(args, fp8rl)
    out.update({"n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "higher_is_better": True,
                "scaling": "weak", "vs_baseline": None, "data": "synthetic"})
    if not args.no_extra:
        extra = {"tiny": tiny(args, fp8rl), "weight_resync": requant(args, fp8rl), "moe_grouped": moe(args, fp8rl),
                 "decode_36_layers": decode(args, fp8rl), "prefill_ue8m0": prefill_ue8m0(args, fp8rl),
                 "dense_mlp": mlp(args, fp8rl),
                 "moe_block": moe_block(args, fp8rl), "tis": tis_step(args, fp8rl),
                 "kv_decode_attention": kv_decode(args, fp8rl),
                 "hbm_copy_GB/s": hbm_copy_reference(),
                 "mfma_probe": mfma_probe(),
                 "operand_streams": dma_probe(args, fp8rl, region_kib=(64, 2048), waves=(8,), inflight=(8,)),
                 "k_step_inner_loop": mfma_loop_probe(args, fp8rl)}
        out["extra"] = extra
        out["roofline"]["frac_of_measured_mfma_loop"] = round(
            out["roofline"]["achieved"] / extra["mfma_probe"]["TFLOP/s"], 4)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(a, w)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
