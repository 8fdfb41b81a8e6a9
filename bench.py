"""Benchmark of the chunkwise GLA forward on one MI355X.

One step = one pass of the hot path over one batch of synthetic input: one
gtr_gla_fwd call (four for the alternating-directions workload, one per scan
direction), with the inputs already resident in HBM when timing starts. The
five workloads of the benchmark are all timed (tiny 16x16 parity case, the
40x40 fp16 operator shape, four directions at 40x40 bf16, 80x80 at chunk 32 / 64
/ 128, a batch of 8 images); the headline line is the 40x40 fp16 operator shape.

Timing protocol (per workload): W eager warm-up steps, then a HIP graph of
G = max(--steps, 100, sets) steps is captured, replayed once untimed, and
replayed 7 times more, each replay bracketed by HIP events on the launch
stream; the figure is the median replay divided by G.
  * cold: the steps rotate over enough distinct device copies of the inputs
    to hold at least 640 MB (2.5x the 256 MB MALL), so every step reads its
    inputs from HBM; the headline value and roofline use this figure;
  * warm: the same input buffers every step.

Prints ONE JSON line. ``roofline`` prices the headline call against HBM
bandwidth with its algorithmic bytes (q, k, g, v in, o out): the whole call is
one launch of the one-launch kernel, so the per-call time is that kernel's
launch duration; ``traffic`` is the HBM traffic per call from the rocprofv3
counter summary under ``profiles/`` (FETCH_SIZE + WRITE_SIZE, scaled by a plain
copy of known size), or null when the kernel sources or the schedule differ
from the ones it was taken on. ``configs`` lists every workload;
``cpu_baseline`` times the float64 oracle on the host on a bounded sample.

``--calibrate-copy MB`` only runs a device-to-device copy of that size (the
reference kernel for the counter scaling) and prints its byte count.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import re
import statistics
import sys
import time

import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import paper_2609_26590_amd as gtr  # noqa: E402
from paper_2609_26590_amd.workloads import (WORKLOADS, algorithmic_bytes, algorithmic_flops,  # noqa: E402
                                            make_inputs, torch_dtype)

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E, published
MFMA_F16_PEAK_TFLOPS = 2500.0  # MI355X dense fp16 matrix, published
KERNEL_SOURCES = ("paper_2609_26590_amd/csrc/gla_fwd.hip", "paper_2609_26590_amd/csrc/gla_lean.hip",
                  "paper_2609_26590_amd/csrc/gla_common.h", "paper_2609_26590_amd/csrc/gtr_device.h")
TRAFFIC_PROFILE = "profiles/gla_kbench_auto_traffic.txt"  # counters of the default (AUTO) run


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def stored_traffic(schedule):
    """HBM bytes per call from the committed counter profile, if it was taken on
    these kernel sources and for this schedule (else None)."""
    path = os.path.join(ROOT, TRAFFIC_PROFILE)
    if not os.path.exists(path):
        return None
    txt = open(path).read()
    m_hash = re.search(r"^kernel source hash:\s*([0-9a-f]+)", txt, re.M)
    m_sched = re.search(r"^schedule:\s*(\w+)", txt, re.M)
    m_val = re.search(r"^traffic bytes per call:\s*([0-9.eE+]+)", txt, re.M)
    if not m_hash or not m_val or not m_sched or m_hash.group(1) != kernel_source_hash() or \
            m_sched.group(1) != schedule:
        return None
    return float(m_val.group(1))


def schedule_of(wl, path):
    """The schedule gtr_gla_fwd runs for the workload (empty tensors of its shapes)."""
    dev = torch.device("cuda")
    mk = lambda d: torch.empty((wl.B, wl.heads, wl.L, d), dtype=torch_dtype(wl.dtype), device=dev)
    s0 = torch.empty((wl.B, wl.heads, wl.dk, wl.dv), device=dev) if wl.s0_std is not None else None
    return gtr.gtr_gla_schedule(mk(wl.dk), mk(wl.dk), mk(wl.dv), mk(wl.dk), H=wl.H, W=wl.W, chunk=wl.chunk,
                                s0=s0, want_final=wl.want_final, o_dtype=torch_dtype(wl.odtype), path=path)


KERNEL_OF = {"inline": "gla_lean_kernel for 16-bit inputs at chunk 64, else gla_chain_kernel (one launch, "
                       "look-back over summaries: the whole call is this kernel)",
             "fused": "gla_lean_kernel for 16-bit inputs at chunk 64, else gla_chain_kernel (one launch, "
                      "look-back to inclusive states: the whole call is this kernel)",
             "staged": "one gtr_gla_fwd call (summary + scan + output kernels)"}


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=100, help="steps per timed graph (at least 100 are captured)")
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--path", default="auto", choices=["auto", "fused", "staged", "inline"])
    p.add_argument("--only", default=None, help="time only these workloads (comma-separated labels)")
    p.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    p.add_argument("--no-cold", action="store_true", help="skip the cold legs")
    p.add_argument("--cpu-seconds", type=float, default=10.0)
    p.add_argument("--detail", action="store_true",
                   help="also time the paper's operator shapes, the fusions and the Spatial SwiGLU")
    p.add_argument("--peaks", action="store_true",
                   help="only measure the achievable copy bandwidth and fp16 GEMM rate and print them")
    p.add_argument("--swiglu-only", action="store_true",
                   help="only time the Spatial SwiGLU (GTR-L and GTR-X widths) and print its JSON line")
    p.add_argument("--block-only", action="store_true",
                   help="only time one GTR block (GTR-S and GTR-L widths, 40x40) and print its JSON line")
    p.add_argument("--calibrate-copy", type=float, default=0.0, metavar="MB",
                   help="only run a device-to-device copy of MB megabytes --steps times")
    return p.parse_args()


def calibrate_copy(mb, steps):
    n = int(mb * 1e6) // 16 * 16
    src = torch.randint(0, 255, (n,), dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        dst.copy_(src)
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "copies": steps,
                      "GBps_read_plus_write": 2 * n * steps / el / 1e9}), flush=True)


COLD_BYTES = 640e6  # input bytes the cold leg rotates over: 2.5x the 256 MB MALL
REPLAYS = 7          # timed replays of each graph; the median is reported


def input_bytes(wl) -> float:
    """Bytes of one input set (q, k, v, g and S0)."""
    es = torch.tensor([], dtype=torch_dtype(wl.dtype)).element_size()
    b = wl.B * wl.heads * wl.L * (3 * wl.dk + wl.dv) * es
    if wl.s0_std is not None:
        b += wl.B * wl.heads * wl.dk * wl.dv * 4
    return float(b)


def setup(wl, path, scans=None, chunk=None, sets=1, fusions=False):
    """A step of the workload (one call per scan direction); call i reads input
    set i % sets. ``fusions``: g holds gate logits (tau = 16) and the
    output-gate epilogue (gate in the input dtype, RMSNorm weight) is fused
    into the store."""
    inp = make_inputs(wl)
    dev = torch.device("cuda")
    extra = {}
    if fusions:
        rng = torch.Generator().manual_seed(wl.seed)
        inp["g"] = (torch.randn(inp["g"].shape, generator=rng) * 2.0).to(torch_dtype(wl.dtype))
        extra = dict(gate_tau=16.0,
                     out_gate=torch.randn((wl.B, wl.heads, wl.L, wl.dv), generator=rng).to(
                         torch_dtype(wl.dtype)).to(dev),
                     norm_weight=torch.rand(wl.dv, generator=rng).to(dev) + 0.5)
    first = {n: (None if inp[n] is None else inp[n].to(dev)) for n in ("q", "k", "v", "g", "s0")}
    # distinct device copies (distinct addresses) of the same values
    copies = [first] + [{n: (None if t is None else t.clone()) for n, t in first.items()} for _ in range(sets - 1)]
    o = torch.empty((wl.B, wl.heads, wl.L, wl.dv), dtype=torch_dtype(wl.odtype), device=dev)
    sf = torch.empty((wl.B, wl.heads, wl.dk, wl.dv), dtype=torch.float32, device=dev) if wl.want_final else None
    ws = gtr.Workspace(dev)
    scans = list(scans or wl.scans)
    C = chunk or wl.chunk

    def step(i=0):
        x = copies[i % sets]
        for scan in scans:
            gtr.gtr_gla_fwd(x["q"], x["k"], x["v"], x["g"], H=wl.H, W=wl.W, scale=wl.scale, chunk=C, scan=scan,
                            s0=x["s0"], out=o, s_final=sf, path=path, workspace=ws, **extra)

    step()  # sizes and zero-fills the workspace outside any capture
    torch.cuda.synchronize()
    return step


def time_graph(step, steps, warmup, replays=REPLAYS):
    """Median seconds per step over `replays` timed replays of a graph of
    `steps` steps (HIP events on the current stream around each replay)."""
    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for i in range(steps):
            step(i)
    graph.replay()  # untimed
    torch.cuda.synchronize()
    times = []
    for _ in range(replays):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        graph.replay()
        e1.record()
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1) / 1000.0 / steps)
    del graph
    torch.cuda.synchronize()
    return statistics.median(times), times


def measure(wl, path, steps, warmup, scans=None, chunk=None, cold=True):
    """(warm, cold) median seconds per step and the cold leg's set count."""
    st = setup(wl, path, scans=scans, chunk=chunk)
    warm, _ = time_graph(st, max(steps, 100), warmup)
    del st
    res = {"warm": warm, "cold": None, "sets": 0}
    if cold:
        sets = max(2, math.ceil(COLD_BYTES / input_bytes(wl)))
        st = setup(wl, path, scans=scans, chunk=chunk, sets=sets)
        res["cold"], _ = time_graph(st, max(steps, 100, sets), warmup)
        res["sets"] = sets
        del st
    torch.cuda.empty_cache()
    return res


def swiglu_detail():
    """Spatial SwiGLU (Sec. 3.1) at the GTR-L and GTR-X widths on the 40x40 grid, fp16."""
    res = {}
    dev = torch.device("cuda")
    for name, d, h in (("swiglu GTR-L d384 h1536", 384, 1536), ("swiglu GTR-X d384 h2304", 384, 2304)):
        gen = torch.Generator().manual_seed(d + h)
        M = 1600
        x = torch.randn((1, M, d), generator=gen).half().to(dev)
        wg = (torch.randn((h, d), generator=gen) * d ** -0.5).half().to(dev)
        wv = (torch.randn((h, d), generator=gen) * d ** -0.5).half().to(dev)
        wo = (torch.randn((d, h), generator=gen) * h ** -0.5).half().to(dev)
        cw = (torch.randn((h, 3, 3), generator=gen) / 3).to(dev)
        cb = (torch.randn(h, generator=gen) * 0.1).to(dev)
        y = torch.empty((1, M, d), dtype=torch.float16, device=dev)
        ws = gtr.Workspace(dev)

        def step(i=0):
            gtr.gtr_spatial_swiglu(x, wg, wv, wo, cw, cb, H=40, W=40, out=y, workspace=ws)

        step()
        torch.cuda.synchronize()
        t, _ = time_graph(step, 100, 10)
        flops = 2.0 * M * d * 2 * h + 2.0 * M * h * d + 18.0 * M * h
        nbytes = M * d * 2 * 2 + 3 * h * d * 2 + h * 40
        res[name] = {"us_per_call": t * 1e6, "tflops": flops / t / 1e12,
                     "mfma_frac": flops / t / 1e12 / MFMA_F16_PEAK_TFLOPS, "alg_GBps": nbytes / t / 1e9}
    return res


def block_detail():
    """One GTR block (Sec. 3.1: projections, GLA with the fused gate and output
    gate, W_o, Spatial SwiGLU, residuals) with random weights on the 40x40 grid,
    fp16, row scan: GTR-S and GTR-L widths. FLOPs: the products (2 M N K each)
    plus the GLA's chunkwise arithmetic."""
    from paper_2609_26590_amd import block
    from paper_2609_26590_amd.workloads import BLOCK_SIZES, make_block
    res = {}
    dev = torch.device("cuda")
    for name in ("gtr_s", "gtr_l"):
        d, heads = BLOCK_SIZES[name]
        x, p = make_block(name, 40, 40)
        x = x.to(dev)
        pd = block.prepare({k: v.to(dev) for k, v in p.items()})

        def step(i=0):
            block.forward(x, pd, H=40, W=40, heads=heads, scan="row")

        step()
        torch.cuda.synchronize()
        t, _ = time_graph(step, 100, 10)
        M, h, dh = 1600, 4 * d, d // heads
        # products: the five-part projection (q, k, v, z, gate logits), W_o, the Spatial SwiGLU's three
        flops = 2.0 * M * (5 * d * d + d * d + 3 * h * d) + heads * M * (2 * dh * 65 + 4 * dh * dh)
        res[f"block {name.upper().replace('_', '-')} d{d} 40x40"] = {
            "us_per_call": t * 1e6, "tflops": flops / t / 1e12, "tokens_per_s": M / t}
    return res


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.lower().startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(wl, budget_s):
    import oracle  # test infrastructure: only this leg of the benchmark uses it
    # the oracle's float64 inputs are prepared once, outside the timed passes
    inp = {n: (None if t is None else t.double().numpy()) for n, t in make_inputs(wl).items()}
    avail = len(os.sched_getaffinity(0))
    threads = max(1, min(avail, wl.B * wl.heads))

    def rate(nthreads, seconds):
        oracle.gla(inp["q"], inp["k"], inp["v"], inp["g"], inp["s0"], scale=wl.scale, H=wl.H, W=wl.W,
                   threads=nthreads)  # load / warm
        reps, t0 = 0, time.perf_counter()
        while True:
            oracle.gla(inp["q"], inp["k"], inp["v"], inp["g"], inp["s0"], scale=wl.scale, H=wl.H, W=wl.W,
                       threads=nthreads)
            reps += 1
            el = time.perf_counter() - t0
            if el >= seconds:
                return reps, el

    reps, el = rate(threads, budget_s * 2 / 3)
    reps1, el1 = rate(1, budget_s / 3)
    tok = wl.B * wl.L  # grid tokens per pass, all heads of each token included, as in `value`
    return {"value": reps * tok / el, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"{reps} full passes of the {wl.name} workload ({wl.B * wl.heads} sequences x {wl.L} "
                      f"tokens, float64 sequential recurrence, sequences spread over the threads; float64 "
                      f"inputs prepared outside the timing) in {el:.1f} s; {reps1} passes on one thread in "
                      f"{el1:.1f} s",
            "single_thread_value": reps1 * tok / el1, "threads_available": avail, "cpu_model": cpu_model()}


def measured_peaks():
    """Achievable rates on this device, for comparison with the published peaks: a 1 GB device-to-device
    copy (HBM read + write) and a large fp16 product through the library GEMM (torch.mm)."""
    n = 1 << 30
    src = torch.empty(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(10):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    copy_gbs = 2 * n * 10 / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del src, dst
    m = 8192
    a = torch.randn((m, m), dtype=torch.float16, device="cuda")
    b = torch.randn((m, m), dtype=torch.float16, device="cuda")
    c = torch.mm(a, b)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(10):
        torch.mm(a, b, out=c)
    e1.record()
    torch.cuda.synchronize()
    mm_tflops = 2.0 * m ** 3 * 10 / (e0.elapsed_time(e1) * 1e-3) / 1e12
    return {"copy_read_plus_write_GBps": copy_gbs, "copy_frac_of_8TBps": copy_gbs / HBM_PEAK_GBS,
            "fp16_gemm_8192_TFLOPs": mm_tflops, "gemm_frac_of_2500": mm_tflops / MFMA_F16_PEAK_TFLOPS}


# The five workloads of the benchmark: (label, workload, scans per step, chunk).
CONFIGS = [
    ("1 tiny", "tiny", None, None),
    ("2 kbench", "kbench", None, None),
    ("3 directions", "directions", ("row", "col", "row_rev", "col_rev"), None),
    ("4 highres C=32", "highres", None, 32),
    ("4 highres C=64", "highres", None, 64),
    ("4 highres C=128", "highres", None, 128),
    ("5 batched", "batched", None, None),
]
HEADLINE = "2 kbench"


def describe(wl, scans, chunk) -> str:
    sc = "/".join(scans) if scans else wl.scans[0]
    extra = ", S0 in, S_final out" if wl.s0_std is not None else ""
    return (f"{wl.name}: B={wl.B} heads={wl.heads} grid {wl.H}x{wl.W} (L={wl.L}) d_k={wl.dk} d_v={wl.dv} "
            f"{wl.dtype} in / {wl.odtype} out, chunk {chunk or wl.chunk}, {sc} scan{extra}")


def config_entry(label, name, scans, chunk, path, steps, warmup, cold):
    wl = WORKLOADS[name]
    if chunk is not None:
        wl = wl.with_(chunk=chunk)
    calls = len(scans) if scans else 1
    r = measure(wl, path, steps, warmup, scans=scans, chunk=chunk, cold=cold)
    t = r["cold"] if r["cold"] is not None else r["warm"]
    per_call = t / calls
    nbytes, flops = algorithmic_bytes(wl), algorithmic_flops(wl)
    e = {"label": label, "workload": describe(wl, scans, chunk), "schedule": schedule_of(wl, path),
         "value_parts": value_parts_of(wl, path), "calls_per_step": calls,
         "us_per_step": t * 1e6, "us_per_call": per_call * 1e6,
         "us_per_call_warm": r["warm"] / calls * 1e6,
         "tokens_per_s": wl.B * wl.L * calls / t, "tflops": flops / per_call / 1e12,
         "alg_bytes_per_call": nbytes, "achieved_GBps": nbytes / per_call / 1e9,
         "hbm_frac": nbytes / per_call / 1e9 / HBM_PEAK_GBS,
         "hbm_frac_warm": nbytes / (r["warm"] / calls) / 1e9 / HBM_PEAK_GBS,
         "timing": "cold" if r["cold"] is not None else "warm"}
    if r["cold"] is not None:
        e["cold_sets"] = r["sets"]
        e["cold_input_MB"] = r["sets"] * input_bytes(wl) / 1e6
    return wl, e


def value_parts_of(wl, path):
    dev = torch.device("cuda")
    mk = lambda d: torch.empty((wl.B, wl.heads, wl.L, d), dtype=torch_dtype(wl.dtype), device=dev)
    s0 = torch.empty((wl.B, wl.heads, wl.dk, wl.dv), device=dev) if wl.s0_std is not None else None
    return gtr.gtr_gla_value_parts(mk(wl.dk), mk(wl.dk), mk(wl.dv), mk(wl.dk), H=wl.H, W=wl.W, chunk=wl.chunk,
                                   s0=s0, want_final=wl.want_final, o_dtype=torch_dtype(wl.odtype), path=path)


def detail(path, steps, warmup):
    """The paper's operator shapes, the fusions and the Spatial SwiGLU (warm)."""
    det = {}
    for name in ("op256", "op1600", "op16k"):
        wl = WORKLOADS[name]
        t, _ = time_graph(setup(wl, path), max(steps, 100), warmup)
        det[name] = {"us_per_call": t * 1e6, "tokens_per_s": wl.B * wl.L / t, "schedule": schedule_of(wl, path),
                     "hbm_frac": algorithmic_bytes(wl) / t / 1e9 / HBM_PEAK_GBS}
    # the same call with gate fusion and the output-gate epilogue (+ the gate input's bytes)
    for name in ("kbench", "op1600", "batched"):
        wl = WORKLOADS[name]
        t, _ = time_graph(setup(wl, path, fusions=True), max(steps, 100), warmup)
        b2 = algorithmic_bytes(wl) + wl.B * wl.heads * wl.L * wl.dv * \
            torch.tensor([], dtype=torch_dtype(wl.dtype)).element_size() + wl.dv * 4
        det[f"{name}+fusions"] = {"us_per_call": t * 1e6, "tokens_per_s": wl.B * wl.L / t,
                                  "hbm_frac": b2 / t / 1e9 / HBM_PEAK_GBS}
    det.update(swiglu_detail())
    det.update(block_detail())
    return det


def main():
    a = parse()
    if a.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; multi-GPU sharding is described in the "
                                   "design notes but not built", "n_gpus": a.gpus}))
        sys.exit(2)
    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(1)
    if a.calibrate_copy > 0:
        calibrate_copy(a.calibrate_copy, a.steps)
        return
    gtr.load()
    if a.swiglu_only:
        print(json.dumps(swiglu_detail()), flush=True)
        return
    if a.block_only:
        print(json.dumps(block_detail()), flush=True)
        return
    if a.peaks:
        print(json.dumps(measured_peaks()), flush=True)
        return
    only = set(x.strip() for x in a.only.split(",")) if a.only else None
    entries, head = [], None
    for label, name, scans, chunk in CONFIGS:
        if only and label not in only and name not in only:
            continue
        wl, e = config_entry(label, name, scans, chunk, a.path, a.steps, a.warmup, cold=not a.no_cold)
        entries.append(e)
        print(f"# {label}: {e['us_per_call']:.2f} us per call ({e['timing']}), {e['us_per_call_warm']:.2f} warm, "
              f"{e['hbm_frac'] * 100:.1f}% of HBM, schedule {e['schedule']}", file=sys.stderr, flush=True)
        if label == HEADLINE:
            head = (wl, e)
    if head is None:
        print(json.dumps({"configs": entries}), flush=True)
        return
    wl, e = head
    per_call = e["us_per_call"] * 1e-6
    G = max(a.steps, 100, e.get("cold_sets", 0))
    out = {
        "metric": "GLA fwd tokens/s and TFLOP/s at 40x40 tokens; % of MFMA/HBM roofline",
        "value": e["tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": G,
        "warmup": a.warmup,
        "ms_per_step": per_call * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic",
        "config": {"workload": e["workload"], "path": a.path,
                   "timing": f"median of {REPLAYS} replays of a {G}-step HIP graph, HIP events on the launch stream; "
                             f"cold: the steps rotate over {e.get('cold_sets')} input sets "
                             f"({e.get('cold_input_MB', 0):.0f} MB, more than the 256 MB MALL)"},
        "token_heads_per_s": wl.B * wl.heads * wl.L / per_call,
        "tflops": e["tflops"],
        "roofline": {"bound": "hbm", "achieved": e["achieved_GBps"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": e["hbm_frac"], "frac_warm": e["hbm_frac_warm"],
                     "traffic": stored_traffic(e["schedule"]),
                     "kernel": KERNEL_OF[e["schedule"]], "schedule": e["schedule"],
                     "alg_bytes_per_call": e["alg_bytes_per_call"], "us_per_call": e["us_per_call"],
                     "us_per_call_warm": e["us_per_call_warm"],
                     "timing": "cold leg: algorithmic bytes per call / median per-call time",
                     "kernel_source_hash": kernel_source_hash(),
                     "mfma_frac": e["tflops"] / MFMA_F16_PEAK_TFLOPS},
        "configs": entries,
    }
    if a.detail:
        out["detail"] = detail(a.path, a.steps, a.warmup)
    elif only is None:
        # the rows beyond the GLA call, timed in every default run: the Spatial
        # SwiGLU and one GTR block (warm, us per image / per block)
        out["beyond_gla"] = {**swiglu_detail(), **block_detail()}
    if not a.no_cpu:
        out["cpu_baseline"] = cpu_baseline(wl, a.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
