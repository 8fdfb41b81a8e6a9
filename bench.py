"""Benchmark of the chunkwise GLA forward on one MI355X.

One step = one gtr_gla_fwd call on the paper's operator-benchmark shape
(B=1, 6 heads, 40x40 token grid -> L=1600, d_k=d_v=64, fp16 in/out, chunk 64,
row-major scan), with inputs already resident in HBM. K steps are captured in
one HIP graph (the paper times its operator under graph replay) and replayed
once inside the timed region.

Prints ONE JSON line (see the keys below). ``roofline`` prices the call's
kernels against HBM bandwidth with the algorithmic bytes of the call;
``cpu_baseline`` times the float64 oracle on the host on a bounded sample of
the same workload. ``roofline.traffic`` is the HBM traffic per call read by
rocprofv3 counters (FETCH_SIZE + WRITE_SIZE, scaled by a plain copy of known
size), taken from the profile summary under ``profiles/``; it is null when the
kernel sources have changed since that summary was written.

``cold`` repeats the timing with the calls rotating over ``--cold-sets``
distinct copies of the inputs (128 copies of 4.9 MB exceed the 256 MB MALL),
so that every call reads its inputs from HBM; the headline ``value`` is the
warm number (the same input buffers every call).

``--calibrate-copy MB`` only runs a device-to-device copy of that size (the
reference kernel for the counter scaling) and prints its byte count.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
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
KERNEL_SOURCES = ("paper_2609_26590_amd/csrc/gla_fwd.hip", "paper_2609_26590_amd/csrc/gtr_device.h")
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


KERNEL_OF = {"inline": "gla_fused_kernel<..., true> (inline schedule; the whole call is this one launch)",
             "fused": "gla_fused_kernel<..., false> (fused schedule; the whole call is this one launch)",
             "staged": "one gtr_gla_fwd call (summary + scan + output kernels)"}


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=500)
    p.add_argument("--warmup", type=int, default=50)
    p.add_argument("--workload", default="kbench", choices=sorted(WORKLOADS))
    p.add_argument("--path", default="auto", choices=["auto", "fused", "staged", "inline"])
    p.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    p.add_argument("--cpu-seconds", type=float, default=10.0)
    p.add_argument("--detail", action="store_true", help="also time the other workloads")
    p.add_argument("--cold-sets", type=int, default=128,
                   help="also time the calls rotating over this many distinct input sets (more bytes than the "
                        "256 MB MALL holds, so every call reads HBM); 0 skips it")
    p.add_argument("--peaks", action="store_true",
                   help="only measure the achievable copy bandwidth and fp16 GEMM rate and print them")
    p.add_argument("--swiglu-only", action="store_true",
                   help="only time the Spatial SwiGLU (GTR-L and GTR-X widths) and print its JSON line")
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


def setup(wl, path, scan=None, sets=1, fusions=False):
    """One call of the workload; ``fusions``: g holds gate logits (tau = 16) and
    the output-gate epilogue (fp16/bf16 gate in the input dtype, RMSNorm weight)
    is fused into the store."""
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
    # `sets` distinct device copies of the inputs; call i reads copy i % sets
    copies = [tuple(inp[n].to(dev) for n in ("q", "k", "v", "g")) for _ in range(sets)]
    s0 = None if inp["s0"] is None else inp["s0"].to(dev)
    o = torch.empty((wl.B, wl.heads, wl.L, wl.dv), dtype=torch_dtype(wl.odtype), device=dev)
    sf = torch.empty((wl.B, wl.heads, wl.dk, wl.dv), dtype=torch.float32, device=dev) if wl.want_final else None
    ws = gtr.Workspace(dev)
    scans = [scan] if scan else list(wl.scans)

    def step(i=0):
        q, k, v, g = copies[i % sets]
        gtr.gtr_gla_fwd(q, k, v, g, H=wl.H, W=wl.W, scale=wl.scale, chunk=wl.chunk, scan=scans[i % len(scans)],
                        s0=s0, out=o, s_final=sf, path=path, workspace=ws, **extra)

    step()  # sizes and zero-fills the workspace outside any capture
    torch.cuda.synchronize()
    return step


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
        t = time_graph(step, 100, 10) / 100
        flops = 2.0 * M * d * 2 * h + 2.0 * M * h * d + 18.0 * M * h
        nbytes = M * d * 2 * 2 + 3 * h * d * 2 + h * 40
        res[name] = {"us_per_call": t * 1e6, "tflops": flops / t / 1e12,
                     "mfma_frac": flops / t / 1e12 / MFMA_F16_PEAK_TFLOPS, "alg_GBps": nbytes / t / 1e9}
    return res


def time_graph(step, steps, warmup):
    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for i in range(steps):
            step(i)
    graph.replay()  # warm replay
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    graph.replay()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / 1000.0  # seconds for `steps` calls


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
    if a.peaks:
        print(json.dumps(measured_peaks()), flush=True)
        return
    wl = WORKLOADS[a.workload]
    sched = schedule_of(wl, a.path)
    step = setup(wl, a.path, scan=wl.scans[0])
    secs = time_graph(step, a.steps, a.warmup)
    per_call = secs / a.steps
    tok_s = wl.B * wl.heads * wl.L / per_call  # token-heads per second
    tokens_s = wl.B * wl.L / per_call          # grid tokens per second (all heads)
    flops = algorithmic_flops(wl)
    nbytes = algorithmic_bytes(wl)
    achieved = nbytes / per_call / 1e9
    out = {
        "metric": "GLA fwd tokens/s and TFLOP/s at 40x40 tokens; % of MFMA/HBM roofline",
        "value": tokens_s,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": per_call * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16" if wl.dtype != "f32" else "f32",
        "data": "synthetic",
        "config": {"workload": f"{wl.name}: B={wl.B} heads={wl.heads} grid {wl.H}x{wl.W} (L={wl.L}) "
                               f"d_k=d_v={wl.dk} {wl.dtype} in / {wl.odtype} out, chunk {wl.chunk}, "
                               f"{wl.scans[0]} scan", "path": a.path, "timing": "HIP graph of K calls"},
        "token_heads_per_s": tok_s,
        "tflops": flops / per_call / 1e12,
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS,
                     "traffic": stored_traffic(sched) if a.workload == "kbench" else None,
                     "kernel": KERNEL_OF[sched], "schedule": sched,
                     "alg_bytes_per_call": nbytes, "us_per_call": per_call * 1e6,
                     "timing": "HIP events around a graph of K calls on the launch stream, divided by K",
                     "kernel_source_hash": kernel_source_hash(),
                     "mfma_frac": flops / per_call / 1e12 / MFMA_F16_PEAK_TFLOPS},
    }
    if a.cold_sets > 1:
        st = setup(wl, a.path, scan=wl.scans[0], sets=a.cold_sets)
        cs = time_graph(st, a.steps, a.warmup) / a.steps
        out["cold"] = {"sets": a.cold_sets, "set_bytes": nbytes - wl.B * wl.heads * wl.L * wl.dv *
                       torch.tensor([], dtype=torch_dtype(wl.odtype)).element_size(),
                       "us_per_call": cs * 1e6, "tokens_per_s": wl.B * wl.L / cs,
                       "achieved_GBps": nbytes / cs / 1e9, "frac": nbytes / cs / 1e9 / HBM_PEAK_GBS}
    if a.detail:
        det = {}
        for name in ("directions", "highres", "batched", "op256", "op1600", "op16k"):
            w2 = WORKLOADS[name]
            for scan in w2.scans:
                st = setup(w2, a.path, scan=scan)
                s2 = time_graph(st, 100, 10) / 100
                det[f"{name}/{scan}"] = {"us_per_call": s2 * 1e6,
                                         "tokens_per_s": w2.B * w2.L / s2,
                                         "GBps": algorithmic_bytes(w2) / s2 / 1e9,
                                         "hbm_frac": algorithmic_bytes(w2) / s2 / 1e9 / HBM_PEAK_GBS}
        # the same call with gate fusion and the output-gate epilogue (+ the gate input's bytes)
        for name in ("kbench", "op1600", "batched"):
            w2 = WORKLOADS[name]
            st = setup(w2, a.path, scan=w2.scans[0], fusions=True)
            s2 = time_graph(st, 100, 10) / 100
            b2 = algorithmic_bytes(w2) + w2.B * w2.heads * w2.L * w2.dv * \
                torch.tensor([], dtype=torch_dtype(w2.dtype)).element_size() + w2.dv * 4
            det[f"{name}+fusions"] = {"us_per_call": s2 * 1e6, "tokens_per_s": w2.B * w2.L / s2,
                                      "GBps": b2 / s2 / 1e9, "hbm_frac": b2 / s2 / 1e9 / HBM_PEAK_GBS}
        out["detail"] = det
    if a.detail:
        out["detail"].update(swiglu_detail())
    if not a.no_cpu:
        out["cpu_baseline"] = cpu_baseline(wl, a.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
