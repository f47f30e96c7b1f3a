"""Benchmark of the fused MoE GEMM2 + combine stage on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload dsv2lite] [--consumers C]
                    [--no-sweep] [--no-cpu] [--calibrate] [--copy-probe MIB]

One step is one call of moe_gemm2_combine (grouped down-projection GEMM plus
the gate-weighted combine, with the launch-time partition selector) on the
DeepSeek-V2-Lite-like one-GPU share (T=16384 tokens, H=2048, I=704, 32 local
experts, top-6, two splits; hottest expert 4x the mean load, the rest Zipf
s=1.2), inputs synthetic and resident in HBM.  Prints one JSON line.

Also measured, in the same run:
  * a trace of one launch (per-tile and per-task timestamps) giving the
    GEMM-portion TFLOP/s and the combine GB/s;
  * the selector sweep: 12 workloads (T in 4096..32768 x uniform / Zipf 0.8 /
    Zipf 1.2 on the same shapes), every consumer count C = 0..64 timed, and
    the selector's pick compared with the best (regret);
  * the CPU oracle on the same workload (the CPU baseline).
"""
from __future__ import annotations

import argparse
import ctypes
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
TICK_S = 1e-8  # the device timestamp runs at 100 MHz


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


class DevWorkload:
    """A workload resident on the GPU, with its workspace."""

    def __init__(self, w, B, torch, synth_tensors=False, seed=0):
        self.w, self.B, self.torch = w, B, torch
        dev = "cuda"
        if synth_tensors:
            # timing-only inputs: same shapes and routing, values drawn on the GPU
            g = torch.Generator(device=dev)
            g.manual_seed(seed)
            self.x = torch.randn((w.Mtot, w.I), generator=g, device=dev).to(torch.bfloat16)
            self.w2 = (torch.randn((w.E, w.I, w.H), generator=g, device=dev)
                       * (1.0 / np.sqrt(w.I))).to(torch.bfloat16)
        else:
            self.x = torch.from_numpy(w.x_perm.view(np.int16)).to(dev).view(torch.bfloat16)
            self.w2 = torch.from_numpy(w.w2.view(np.int16)).to(dev).view(torch.bfloat16)
        self.off = torch.from_numpy(w.expert_offsets).to(dev)
        self.tid = torch.from_numpy(w.token_ids).to(dev)
        self.g = torch.from_numpy(w.gate_w).to(dev)
        self.out = torch.empty((w.T, w.H), dtype=torch.float32, device=dev)
        self.wl, self._keep = B.make_workload(w.T, w.H, w.I, w.E, w.topk, w.L, w.counts)
        self.ws = B.Workspace(B.workspace_size(self.wl))

    def run(self, C=-1, trace=None, mode=None):
        """One launch; mode None is moe_gemm2_combine (owner-write), 0/1 go
        through moe_gemm2_combine_ex."""
        w = self.w
        return self.B.combine(self.x, self.w2, self.off, self.tid, self.g, T=w.T, splits=w.L,
                              topk=w.topk, counts=w.counts, num_consumers=C, out=self.out,
                              workspace=self.ws, trace=trace, mode=mode)[1]

    def trace(self, C, mode=None):
        """One traced launch: (C used, tiles [n,4], tasks [m,4]) timestamps."""
        torch, B, w = self.torch, self.B, self.w
        buf = torch.zeros(B.trace_size(self.wl) // 8, dtype=torch.int64, device="cuda")
        used = self.run(C, trace=buf, mode=mode)
        torch.cuda.synchronize()
        tr = buf.cpu().numpy().astype(np.int64)
        part = B.select_partition(self.wl, B.launch_params(self.wl, mode or 0))[1]
        n_tiles = int(part.W_comp) * w.L
        ntasks = n_tiles if mode == 1 else int(part.W_comm) * w.L
        # tile records first (room for max_tiles), then the task records
        max_tiles = w.L * (-(-(w.H // w.L) // 256)) * (-(-w.Mtot // 256) + w.E)
        tiles = tr[: 4 * n_tiles].reshape(-1, 4)
        tasks = tr[4 * max_tiles: 4 * (max_tiles + ntasks)].reshape(-1, 4)
        return used, tiles, tasks


def breakdown(dw, C, mode=None, reps=5):
    """GEMM portion and combine from traced launches: the launch with the
    median GEMM span out of `reps` (each after a short pause, so that one
    launch's clock state does not decide the figure)."""
    w = dw.w
    flops, gemm_bytes, combine_bytes, _ = algorithmic(w)
    runs = []
    for _ in range(reps):
        time.sleep(0.05)
        used, tiles, tasks = dw.trace(C, mode)
        runs.append((tiles[:, 3].max() - tiles[:, 0].min(), used, tiles, tasks))
    runs.sort(key=lambda r: r[0])
    _, used, tiles, tasks = runs[len(runs) // 2]
    if mode == 1:   # Y read, ids and gates, one fp32 atomic per routed element, zeroing
        combine_bytes = w.Mtot * w.H * 2 + w.Mtot * 8 + w.Mtot * w.H * 4 + w.T * w.H * 4
    gemm_span = (tiles[:, 3].max() - tiles[:, 0].min()) * TICK_S
    gp = {"span_us": gemm_span * 1e6, "tflops": flops / gemm_span / 1e12,
          "pct_peak": 100 * flops / gemm_span / 1e12 / PEAK_BF16_TFLOPS,
          "mean_tile_us": float((tiles[:, 3] - tiles[:, 0]).mean() * TICK_S * 1e6),
          "mean_reduction_loop_us": float((tiles[:, 1] - tiles[:, 0]).mean() * TICK_S * 1e6),
          "mean_store_publish_us": float((tiles[:, 3] - tiles[:, 1]).mean() * TICK_S * 1e6)}
    comb = None
    if len(tasks) and tasks[:, 2].max() > 0:
        busy = tasks[:, 2] - tasks[:, 1]
        cspan = (tasks[:, 2].max() - tasks[:, 1].min()) * TICK_S
        comb = {"span_us": cspan * 1e6, "gbps": combine_bytes / cspan / 1e9,
                "mean_task_us": float(busy.mean() * TICK_S * 1e6),
                "tail_after_gemm_us": float((tasks[:, 2].max() - tiles[:, 3].max()) * TICK_S * 1e6)}
    return used, gp, comb


def calibrate(dw, C_ref=32, reps=5, mode=None):
    """rho_ref: one consumer-task wave over one compute-tile wave, measured at
    a fixed consumer count (the paper's calibration procedure)."""
    task_t, tile_t = [], []
    for _ in range(reps):
        _, tiles, tasks = dw.trace(C_ref, mode)
        tile_t.append((tiles[:, 3] - tiles[:, 0]).mean())
        task_t.append((tasks[:, 2] - tasks[:, 1]).mean())
    tile_us = float(np.median(tile_t)) * TICK_S * 1e6
    task_us = float(np.median(task_t)) * TICK_S * 1e6
    return {"C_ref": C_ref, "compute_wave_us": round(tile_us, 3),
            "consumer_wave_us": round(task_us, 3), "rho_ref": round(task_us / tile_us, 4)}


def time_launches(dw, Cs, samples, torch):
    """Median event time per C, samples interleaved forward/backward (ABBA).
    A C may be a (C, mode) pair to time moe_gemm2_combine_ex in that mode."""
    stream = torch.cuda.current_stream()
    times = {C: [] for C in Cs}

    def launch(C):
        return dw.run(C[0], mode=C[1]) if isinstance(C, tuple) else dw.run(C)

    for C in Cs:               # warm-up of every partition
        launch(C)
    torch.cuda.synchronize()
    for s in range(samples):
        order = list(Cs) if s % 2 == 0 else list(reversed(Cs))
        evs = []
        for C in order:
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            launch(C)
            b.record(stream)
            evs.append((C, a, b))
        torch.cuda.synchronize()
        for C, a, b in evs:
            times[C].append(a.elapsed_time(b))
    return {C: float(np.median(v)) for C, v in times.items()}


def run_sweep(B, torch, samples, c_max=64):
    """Time every C in 0..c_max on the 12 sweep workloads; compare the
    selector's pick with the fastest (regret = (t_pick - t_best) / t_best).
    The library's candidate set is 0..64 (C = 0: role switch); the paper's
    legal set is 1..C_max, reported separately."""
    from workloads import sweep_workload, sweep_workloads
    base_params = B.default_params(0)
    rows = []
    for name, _ in sweep_workloads():
        w = sweep_workload(name, with_tensors=False)
        log(f"sweep {name}: rows={w.Mtot} r_expert={w.r_expert:.2f}")
        dw = DevWorkload(w, B, torch, synth_tensors=True)
        params = B.launch_params(dw.wl)        # what a launch with C = -1 uses
        params_paper = B.launch_params(dw.wl)
        params_paper.c_min = 1
        Cs = list(range(0, c_max + 1))
        med = time_launches(dw, Cs, samples, torch)
        best_all = min(Cs, key=lambda c: med[c])
        best_dom = min(Cs[1:], key=lambda c: med[c])
        pick = B.select_partition(dw.wl, params)[0]
        pick_p = B.select_partition(dw.wl, params_paper)[0]
        # the selector without the routed counts (even-load estimate), as a
        # launch that reads nothing back from the device would run it
        wl_est, _ = B.make_workload(w.T, w.H, w.I, w.E, w.topk, w.L, None)
        pick_e = B.select_partition(wl_est, B.launch_params(wl_est))[0]
        rows.append({
            "workload": name, "T": w.T, "r_expert": round(w.r_expert, 3),
            "task_tokens": params.comm_tile_m,
            "best_C": best_all, "best_us": round(med[best_all] * 1e3, 1),
            "pick_C": pick, "pick_us": round(med[pick] * 1e3, 1),
            "regret": round((med[pick] - med[best_all]) / med[best_all], 4),
            "pick_C_estimate": pick_e, "pick_us_estimate": round(med[pick_e] * 1e3, 1),
            "regret_estimate": round((med[pick_e] - med[best_all]) / med[best_all], 4),
            "best_C_1_64": best_dom, "best_us_1_64": round(med[best_dom] * 1e3, 1),
            "pick_C_paper_set": pick_p, "pick_us_paper_set": round(med[pick_p] * 1e3, 1),
            "regret_paper_set_vs_best_1_64": round((med[pick_p] - med[best_dom]) / med[best_dom], 4),
            "us_by_C": {str(c): round(med[c] * 1e3, 1) for c in Cs},
        })
        del dw
        torch.cuda.empty_cache()

    def agg(key):
        v = [r[key] for r in rows]
        return {"mean": round(float(np.mean(v)), 4), "max": round(float(np.max(v)), 4)}

    return {"workloads": len(rows), "samples_per_C": samples, "C_range": [0, c_max],
            "rho_ref_64_token_task": [base_params.rho_ref_num, base_params.rho_ref_den],
            "regret": agg("regret"),
            "regret_estimate": agg("regret_estimate"),
            "regret_paper_set_vs_best_1_64": agg("regret_paper_set_vs_best_1_64"),
            "per_workload": rows}


def layer_measure(dw, B, torch, samples=20):
    """The whole post-router layer on the same routing: the up-projection
    (grouped GEMM1 + SwiGLU, moe_gemm1_swiglu), the layer (moe_layer_forward)
    and this stage alone, launch for launch interleaved; the stage's share of
    the layer is the quantity the paper reports for its baseline."""
    w = dw.w
    g = torch.Generator(device="cuda")
    g.manual_seed(1)
    hidden = torch.randn((w.T, w.H), generator=g, device="cuda").to(torch.bfloat16)
    w1 = (torch.randn((w.E, w.H, 2 * w.I), generator=g, device="cuda")
          * (1.0 / np.sqrt(w.H))).to(torch.bfloat16)
    w1p = B.pack_w1(w1)
    del w1
    xbuf = torch.empty((w.Mtot, w.I), dtype=torch.bfloat16, device="cuda")
    out = torch.empty((w.T, w.H), dtype=torch.float32, device="cuda")
    wl, _keep = B.make_workload(w.T, w.H, w.I, w.E, w.topk, w.L, w.counts, rows=w.Mtot)
    lws = B.Workspace(B.layer_workspace_size(wl))

    def gemm1():
        B.gemm1_swiglu(hidden, w1p, dw.off, dw.tid, topk=w.topk, rows=w.Mtot, counts=w.counts,
                       out=xbuf, workspace=dw.ws)

    def layer():
        B.layer_forward(hidden, w1p, dw.w2, dw.off, dw.tid, dw.g, topk=w.topk, splits=w.L,
                        counts=w.counts, out=out, workspace=lws)

    fns = {"gemm1": gemm1, "layer": layer, "stage": lambda: dw.run(-1)}
    for f in fns.values():
        f()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    times = {k: [] for k in fns}
    keys = list(fns)
    for s in range(samples):
        order = keys if s % 2 == 0 else keys[::-1]
        evs = []
        for k in order:
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            fns[k]()
            b.record(stream)
            evs.append((k, a, b))
        torch.cuda.synchronize()
        for k, a, b in evs:
            times[k].append(a.elapsed_time(b) * 1e3)
    assert dw.ws.status() == 0 and lws.status() == 0
    med = {k: float(np.median(v)) for k, v in times.items()}
    f1 = 2 * w.Mtot * w.H * 2 * w.I
    f2 = 2 * w.Mtot * w.I * w.H
    return {"us_gemm1_swiglu": round(med["gemm1"], 1),
            "gemm1_tflops": round(f1 / med["gemm1"] / 1e6, 1),
            "us_layer": round(med["layer"], 1),
            "layer_tflops": round((f1 + f2) / med["layer"] / 1e6, 1),
            "us_gemm2_combine": round(med["stage"], 1),
            "gemm2_combine_share_of_layer": round(med["stage"] / med["layer"], 4),
            "samples": samples,
            "inputs": "hidden N(0,1) and W1 N(0,1/H) drawn on the GPU, the stage's routing"}


def spread(samples_us, reps=2000, seed=0):
    """Median, p10/p90 and a bootstrap 95% confidence interval of the median."""
    v = np.asarray(samples_us, dtype=np.float64)
    rng = np.random.default_rng(seed)
    meds = np.median(v[rng.integers(0, len(v), size=(reps, len(v)))], axis=1)
    return {"median": round(float(np.median(v)), 2), "p10": round(float(np.percentile(v, 10)), 2),
            "p90": round(float(np.percentile(v, 90)), 2),
            "ci95_median": [round(float(np.percentile(meds, 2.5)), 2),
                            round(float(np.percentile(meds, 97.5)), 2)],
            "samples": int(len(v))}


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
    return {"value": round(flops / per / 1e12, 4), "unit": "TFLOP/s", "cores": int(threads),
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
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--sweep-samples", type=int, default=7)
    ap.add_argument("--calibrate", action="store_true",
                    help="print the rho_ref calibration at C=32 (both consumer modes) and exit")
    ap.add_argument("--no-layer", action="store_true",
                    help="skip the whole-layer measurement (up-projection + this stage)")
    ap.add_argument("--no-scatter", action="store_true",
                    help="skip the comparison with the atomic-scatter consumer mode")
    ap.add_argument("--timed-only", action="store_true",
                    help="only the warm-up and the timed steps (for profiler runs): no cold-cache "
                         "samples, trace, scatter comparison, sweep or CPU baseline")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run 3 device copies of MIB MiB (HBM counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this stage runs on one GPU; multi-GPU runs are not "
                          "supported (use --gpus 1)"}))
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
    log(f"generating workload {args.workload}")
    w = config(args.workload)
    dw = DevWorkload(w, B, torch)
    if args.calibrate:
        dw.run(32)
        dw.run(32, mode=1)
        torch.cuda.synchronize()
        print(json.dumps({"calibration": calibrate(dw),
                          "calibration_scatter": calibrate(dw, mode=1),
                          "kernel_sha": kernel_sha()}), flush=True)
        return
    stream = torch.cuda.current_stream()

    log("warmup")
    C_used = dw.run(args.consumers)
    for _ in range(args.warmup):
        dw.run(args.consumers)
    torch.cuda.synchronize()
    st = dw.ws.status()
    assert st == 0, B.strerror(st)

    # selector cost on the host (pure C++, no HIP calls), 10^5 calls through
    # ctypes; the same loop around a call that does nothing (the ABI version)
    # gives the ctypes overhead, which the net figure leaves out
    params = B.launch_params(dw.wl)
    L_ = B.lib()
    nsel = 100000
    sel_fn, nop_fn = L_.moe_select_partition, L_.moe_gemm2_abi_version
    wl_ref, p_ref = ctypes.byref(dw.wl), ctypes.byref(params)
    t0 = time.perf_counter()
    for _ in range(nsel):
        sel_fn(wl_ref, p_ref, None)
    sel_us = (time.perf_counter() - t0) / nsel * 1e6
    t0 = time.perf_counter()
    for _ in range(nsel):
        nop_fn()
    nop_us = (time.perf_counter() - t0) / nsel * 1e6

    log(f"timing {args.steps} steps, C={C_used}")
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        starts[i].record(stream)
        dw.run(args.consumers)
        ends[i].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ker_ms = np.array([s.elapsed_time(e) for s, e in zip(starts, ends)])
    ms_per_step = wall * 1e3 / args.steps
    ker_avg_s = float(ker_ms.mean()) / 1e3

    flops, gemm_bytes, combine_bytes, min_bytes = algorithmic(w)
    tflops = flops / (ms_per_step / 1e3) / 1e12
    achieved = flops / ker_avg_s / 1e12

    if args.timed_only:
        print(json.dumps({"metric": METRIC, "value": round(tflops, 2), "unit": "TFLOP/s",
                          "ms_per_step": round(ms_per_step, 4),
                          "avg_launch_us": round(ker_avg_s * 1e6, 2),
                          "us_per_layer": round(float(np.median(ker_ms)) * 1e3, 2),
                          "kernel_sha": kernel_sha()}), flush=True)
        return
    # cold-cache latency: 512 MiB scratch write between samples (untimed)
    scratch = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    cold = []
    for i in range(10):
        scratch.fill_(i)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        dw.run(args.consumers)
        b.record(stream)
        torch.cuda.synchronize()
        cold.append(a.elapsed_time(b))
    del scratch

    _, gemm_portion, combine = breakdown(dw, C_used)
    st = dw.ws.status()
    assert st == 0, B.strerror(st)

    scatter = None
    if not args.no_scatter:
        # the atomic-scatter consumer (mode 1) against the owner-write one,
        # launch for launch (ABBA), each with the selector's pick and C = 0
        log("owner-write vs atomic scatter")
        C_sc = dw.run(-1, mode=1)
        torch.cuda.synchronize()
        keys = sorted({(C_used, 0), (0, 0), (C_sc, 1), (0, 1)})
        med = time_launches(dw, keys, 15, torch)
        st = dw.ws.status()
        assert st == 0, B.strerror(st)
        _, gp_sc, comb_sc = breakdown(dw, C_sc, mode=1)
        scatter = {"selector_C": C_sc,
                   "us_per_layer": {f"mode{m}_C{c}": round(v * 1e3, 1)
                                    for (c, m), v in med.items()},
                   "scatter_over_owner_write": round(med[(C_sc, 1)] / med[(C_used, 0)], 4),
                   "gemm_portion": {k: round(v, 3) for k, v in gp_sc.items()},
                   "combine": {k: round(v, 3) for k, v in comb_sc.items()} if comb_sc else None}

    layer_res = None
    if not args.no_layer:
        log("post-router layer")
        layer_res = layer_measure(dw, B, torch)

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
        "us_per_layer_stats": spread(ker_ms * 1e3),
        "us_per_layer_cold_stats": spread(np.asarray(cold) * 1e3),
        "pct_bf16_peak": round(100 * tflops / PEAK_BF16_TFLOPS, 2),
        "consumers": C_used,
        "selector_us": round(sel_us, 3),
        "selector_us_net_of_ctypes": round(max(sel_us - nop_us, 0.0), 3),
        "gemm_portion": {k: round(v, 3) for k, v in gemm_portion.items()},
        "combine": {k: round(v, 3) for k, v in combine.items()} if combine else None,
        "scatter_mode": scatter,
        "layer": layer_res,
        "roofline": {"bound": "mfma", "achieved": round(achieved, 2),
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": traffic_entry(w.name),
                     "kernel": KERNEL_NAME, "kernel_sha": kernel_sha(),
                     "avg_launch_us": round(ker_avg_s * 1e6, 2),
                     "algorithmic_flops_per_launch": flops,
                     "hbm_bytes_lower_bound": min_bytes,
                     "hbm_bytes_with_y_staging": gemm_bytes + combine_bytes},
    }
    if not args.no_sweep:
        del dw
        torch.cuda.empty_cache()
        log("selector sweep")
        res["sweep"] = run_sweep(B, torch, args.sweep_samples)
    if not args.no_cpu:
        log("timing the CPU oracle")
        res["cpu_baseline"] = cpu_baseline(w)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
