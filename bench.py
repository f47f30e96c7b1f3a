"""Benchmark of the fused MoE GEMM2 + combine stage on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload dsv2lite] [--consumers C]
                    [--sweep] [--no-cpu]

One step is one call of moe_gemm2_combine (grouped down-projection GEMM plus
the gate-weighted combine, with the launch-time partition selector) on the
DeepSeek-V2-Lite-like one-GPU share (T=16384 tokens, H=2048, I=704, 32 local
experts, top-6, two splits; hottest expert 4x the mean load, the rest Zipf
s=1.2), inputs synthetic and resident in HBM.  Prints one JSON line.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "GEMM2+combine µs/layer & TFLOP/s (% bf16 peak); selector regret vs sweep"
PEAK_BF16_TFLOPS = 2500.0
PEAK_HBM_GBS = 8000.0
KERNEL_NAME = "moe_gemm2_fused"
KERNEL_SRC = os.path.join(ROOT, "paper_2609_07536_amd", "csrc", "moe_gemm2.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_moe_gemm2_fused_dsv2lite.json")


def kernel_sha() -> str:
    with open(KERNEL_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def algorithmic(w):
    flops = 2 * w.Mtot * w.I * w.H
    gemm_bytes = w.Mtot * w.I * 2 + w.E * w.I * w.H * 2 + w.Mtot * w.H * 2
    combine_bytes = w.Mtot * w.H * 2 + w.Mtot * 8 + w.T * w.H * 4
    min_bytes = w.Mtot * w.I * 2 + w.E * w.I * w.H * 2 + w.Mtot * 8 + w.T * w.H * 4
    return flops, gemm_bytes, combine_bytes, min_bytes


def traffic_entry(workload_name):
    """HBM bytes per launch from the committed rocprofv3 counter summary,
    only while the kernel source is the one the counters were taken on."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel_sha") != kernel_sha() or t.get("workload") != workload_name:
        return None
    return t.get("hbm_bytes_per_launch")


def cpu_baseline(w, budget_s=12.0):
    """The oracle as it stands, timed on the host cores on this workload."""
    import threadpoolctl
    from oracle import combine as oc
    info = threadpoolctl.threadpool_info()
    threads = max([i.get("num_threads", 1) for i in info if i.get("user_api") == "blas"],
                  default=1)
    n = 0
    t0 = time.perf_counter()
    while True:
        oc.combine_reference(w.x_perm, w.w2, w.expert_offsets, w.token_ids, w.gate_w, w.T)
        n += 1
        el = time.perf_counter() - t0
        if el >= budget_s or n >= 20:
            break
    per = el / n
    flops = 2 * w.Mtot * w.I * w.H
    return {"value": flops / per / 1e12, "unit": "TFLOP/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"whole {w.name} workload (numpy fp32 per-expert matmul + per-token "
                      f"weighted sum), {n} run(s), {per * 1e3:.1f} ms each; "
                      f"host os.cpu_count()={os.cpu_count()}"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="dsv2lite")
    ap.add_argument("--consumers", type=int, default=-1)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--sweep", action="store_true",
                    help="also time C = 0..64 on the 12 sweep workloads (selector regret)")
    ap.add_argument("--sweep-samples", type=int, default=15)
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run 3 device copies of MIB MiB (HBM counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this stage runs on one GPU; multi-GPU runs are not "
                          "part of this build (use --gpus 1)"}))
        sys.exit(2)

    import torch
    from paper_2609_07536_amd import binding as B
    from workloads import CONFIG_TITLES, config

    assert torch.cuda.is_available(), "bench needs a GPU"
    if args.copy_probe:
        n = args.copy_probe << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": n, "copies": 3}), flush=True)
        return
    B.lib()
    dev = "cuda"
    log(f"generating workload {args.workload}")
    w = config(args.workload)
    x = torch.from_numpy(w.x_perm.view(np.int16)).to(dev).view(torch.bfloat16)
    w2 = torch.from_numpy(w.w2.view(np.int16)).to(dev).view(torch.bfloat16)
    off = torch.from_numpy(w.expert_offsets).to(dev)
    tid = torch.from_numpy(w.token_ids).to(dev)
    g = torch.from_numpy(w.gate_w).to(dev)
    out = torch.empty((w.T, w.H), dtype=torch.float32, device=dev)
    wl, keep = B.make_workload(w.T, w.H, w.I, w.E, w.topk, w.L, w.counts)
    ws = B.Workspace(B.workspace_size(wl))
    stream = torch.cuda.current_stream()

    def step(C=args.consumers):
        return B.combine(x, w2, off, tid, g, T=w.T, splits=w.L, topk=w.topk,
                         counts=w.counts, num_consumers=C, out=out, workspace=ws)[1]

    log("warmup")
    C_used = step()
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    st = ws.status()
    assert st == 0, B.strerror(st)

    # selector cost on the host (pure C++, no HIP calls)
    params = B.default_params(0)
    t0 = time.perf_counter()
    nsel = 20000
    for _ in range(nsel):
        B.lib().moe_select_partition(wl, params, None)
    sel_us = (time.perf_counter() - t0) / nsel * 1e6

    log(f"timing {args.steps} steps, C={C_used}")
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        starts[i].record(stream)
        step()
        ends[i].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ker_ms = np.array([s.elapsed_time(e) for s, e in zip(starts, ends)])
    ms_per_step = wall * 1e3 / args.steps
    ker_avg_s = float(ker_ms.mean()) / 1e3

    flops, gemm_bytes, combine_bytes, min_bytes = algorithmic(w)
    tflops = flops / (ms_per_step / 1e3) / 1e12
    achieved = flops / ker_avg_s / 1e12

    # cold-cache latency: 512 MiB scratch write between samples (untimed)
    scratch = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    cold = []
    for i in range(10):
        scratch.fill_(i)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        step()
        b.record(stream)
        torch.cuda.synchronize()
        cold.append(a.elapsed_time(b))
    del scratch

    # one traced launch: split the span into the compute role and the consumers
    trace = torch.zeros(B.trace_size(wl) // 8, dtype=torch.int64, device=dev)
    B.combine(x, w2, off, tid, g, T=w.T, splits=w.L, topk=w.topk, counts=w.counts,
              num_consumers=C_used, out=out, workspace=ws, trace=trace)
    torch.cuda.synchronize()
    tr = trace.cpu().numpy().astype(np.int64)
    part = B.select_partition(wl, params)[1]
    n_tiles = int(part.W_comp) * w.L
    tiles = tr[: 4 * n_tiles].reshape(-1, 4)[:, [0, 3]]
    ntasks = int(part.W_comm) * w.L
    tasks = tr[len(tr) - 4 * ntasks:].reshape(-1, 4) if ntasks else None
    tick = 1e-8  # 100 MHz
    gemm_span = (tiles[:, 1].max() - tiles[:, 0].min()) * tick
    gemm_portion = {"span_us": gemm_span * 1e6, "tflops": flops / gemm_span / 1e12,
                    "pct_peak": 100 * flops / gemm_span / 1e12 / PEAK_BF16_TFLOPS,
                    "mean_tile_us": float((tiles[:, 1] - tiles[:, 0]).mean() * tick * 1e6)}
    combine = None
    if tasks is not None and tasks[:, 2].max() > 0:
        busy = tasks[:, 2] - tasks[:, 1]
        cspan = (tasks[:, 2].max() - tasks[:, 1].min()) * tick
        combine = {"span_us": cspan * 1e6, "gbps": combine_bytes / cspan / 1e9,
                   "mean_task_us": float(busy.mean() * tick * 1e6),
                   "tail_after_gemm_us": float((tasks[:, 2].max() - tiles[:, 1].max()) * tick * 1e6)}

    res = {
        "metric": METRIC,
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": CONFIG_TITLES.get(w.name, w.name), "T": w.T, "H": w.H,
                   "I": w.I, "E": w.E, "topk": w.topk, "splits": w.L,
                   "routed_rows": w.Mtot, "r_expert": round(w.r_expert, 3),
                   "parallelism": "single GPU"},
        "us_per_layer": round(float(np.median(ker_ms)) * 1e3, 2),
        "us_per_layer_cold": round(float(np.median(cold)) * 1e3, 2),
        "pct_bf16_peak": round(100 * tflops / PEAK_BF16_TFLOPS, 2),
        "consumers": C_used,
        "selector_us": round(sel_us, 3),
        "gemm_portion": {k: round(v, 3) for k, v in gemm_portion.items()},
        "combine": {k: round(v, 3) for k, v in combine.items()} if combine else None,
        "roofline": {"bound": "mfma", "achieved": round(achieved, 2),
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": traffic_entry(w.name),
                     "kernel": KERNEL_NAME, "kernel_sha": kernel_sha(),
                     "avg_launch_us": round(ker_avg_s * 1e6, 2)},
    }
    if args.sweep:
        from paper_2609_07536_amd import sweep as S
        res["sweep"] = S.run_sweep(samples=args.sweep_samples, log=log)
    if not args.no_cpu:
        log("timing the CPU oracle")
        res["cpu_baseline"] = cpu_baseline(w)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
