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
        # sized for every split count up to 8 (token-band sweeps vary L)
        wl8, _ = B.make_workload(w.T, w.H, w.I, w.E, w.topk, 8, w.counts)
        self.ws = B.Workspace(max(B.workspace_size(self.wl), B.workspace_size(wl8)))

    def workload(self, splits=None):
        return self.B.make_workload(self.w.T, self.w.H, self.w.I, self.w.E, self.w.topk,
                                    splits or self.w.L, self.w.counts)

    def run(self, C=-1, trace=None, mode=None, splits=None):
        """One launch; mode None is moe_gemm2_combine (owner-write, column
        splits), 0/1/2 go through moe_gemm2_combine_ex."""
        w = self.w
        return self.B.combine(self.x, self.w2, self.off, self.tid, self.g, T=w.T,
                              splits=splits or w.L, topk=w.topk, counts=w.counts,
                              num_consumers=C, out=self.out, workspace=self.ws, trace=trace,
                              mode=mode)[1]

    def trace(self, C, mode=None, splits=None):
        """One traced launch: (C used, tiles [n,4], tasks [m,4]) timestamps
        (tile records in global tile order, task records in task order)."""
        torch, B, w = self.torch, self.B, self.w
        L = splits or w.L
        wl, _keep = self.workload(L)
        buf = torch.zeros(B.trace_size(wl) // 8, dtype=torch.int64, device="cuda")
        used = self.run(C, trace=buf, mode=mode, splits=L)
        torch.cuda.synchronize()
        tr = buf.cpu().numpy().astype(np.int64)
        max_tiles = L * (-(-(-(-w.H // L)) // 256)) * (-(-w.Mtot // 256) + w.E)
        tiles = tr[: 4 * max_tiles].reshape(-1, 4)
        n_tiles = int(np.flatnonzero(tiles[:, 3])[-1]) + 1 if tiles[:, 3].any() else 0
        tiles = tiles[:n_tiles]
        tasks = tr[4 * max_tiles:].reshape(-1, 4)
        n_tasks = int(np.flatnonzero(tasks[:, 2])[-1]) + 1 if tasks[:, 2].any() else 0
        tasks = tasks[:n_tasks]
        return used, tiles, tasks


def settle_calls(fns, torch, ms=60.0, rounds=4):
    """Untimed back-to-back calls of `fns` (in turn, `rounds` each between
    synchronisations) for `ms` of wall time: after an idle period the GPU's
    first ~15 ms of sustained load run slow (on the DeepSeek-V2-Lite-like
    share the first ~40 launches 5-10% above the steady state), so timed
    launches right after one would measure the clock's ramp rather than
    the kernels.  Returns the number of calls."""
    n = 0
    t0 = time.perf_counter()
    while True:
        for _ in range(rounds):
            for f in fns:
                f()
                n += 1
        torch.cuda.synchronize()
        if (time.perf_counter() - t0) * 1e3 >= ms:
            return n


def settle(dw, C, torch, ms=60.0):
    """The settle phase before the timed steps (see settle_calls)."""
    return settle_calls([lambda: dw.run(C)], torch, ms, rounds=16)


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


def task_busy(dw, tasks, mode=None):
    """Busy time of each traced consumer task, in ticks, scaled to the
    launch's comm_tile_m tokens: owner-write tasks of the last split hold
    comm_tile_m_last tokens, and a task's work is proportional to its tokens
    (the assumption rho's scaling makes)."""
    busy = (tasks[:, 2] - tasks[:, 1]).astype(np.float64)
    if mode in (None, 0):
        p = dw.B.launch_params(dw.wl)
        tm, tm_last = p.comm_tile_m, p.comm_tile_m_last or p.comm_tile_m
        if tm_last != tm:
            tps = -(-dw.w.T // tm) * -(-(-(-dw.w.H // dw.w.L)) // 1024)
            busy[(dw.w.L - 1) * tps:] *= tm / tm_last
    return busy


def calibrate(dw, C_ref=32, reps=5, mode=None):
    """rho_ref: one consumer-task wave over one compute-tile wave, measured at
    a fixed consumer count (the paper's calibration procedure)."""
    task_t, tile_t = [], []
    for _ in range(reps):
        _, tiles, tasks = dw.trace(C_ref, mode)
        tile_t.append((tiles[:, 3] - tiles[:, 0]).mean())
        task_t.append(task_busy(dw, tasks, mode).mean())
    tile_us = float(np.median(tile_t)) * TICK_S * 1e6
    task_us = float(np.median(task_t)) * TICK_S * 1e6
    return {"C_ref": C_ref, "compute_wave_us": round(tile_us, 3),
            "consumer_wave_us": round(task_us, 3), "rho_ref": round(task_us / tile_us, 4)}


def time_launches(dw, Cs, samples, torch, warmups=1):
    """Median event time per configuration (ms), samples interleaved
    forward/backward (ABBA).  A configuration is C, or (C, mode) to time
    moe_gemm2_combine_ex in that mode, or (C, mode, splits)."""
    t = time_configs(lambda c: launch_cfg(dw, c), list(Cs), samples, warmups, torch)
    return {c: float(np.median(v)) / 1e3 for c, v in t.items()}


def launch_cfg(dw, c):
    if isinstance(c, tuple):
        return dw.run(c[0], mode=c[1], splits=c[2] if len(c) > 2 else None)
    return dw.run(c)


def time_configs(launch, keys, samples, warmups, torch):
    """Event time (us) of every key, `samples` times each: a settle phase
    (settle_calls) and `warmups` untimed passes over all keys, then passes
    alternately forward and backward over the keys (ABBA), one stream
    synchronisation per pass.  Each pass starts with an untimed launch of
    its first key, so that no timed launch starts on a GPU left idle by the
    synchronisation."""
    stream = torch.cuda.current_stream()
    settle_calls([lambda k=k: launch(k) for k in keys], torch, rounds=1)
    for _ in range(warmups):
        for k in keys:
            launch(k)
    torch.cuda.synchronize()
    times = {k: [] for k in keys}
    for s in range(samples):
        order = keys if s % 2 == 0 else keys[::-1]
        launch(order[0])
        evs = []
        for k in order:
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            launch(k)
            b.record(stream)
            evs.append((k, a, b))
        torch.cuda.synchronize()
        for k, a, b in evs:
            times[k].append(a.elapsed_time(b) * 1e3)
    return times


def median_ci(v, reps=1000, seed=0):
    """Median and a bootstrap 95% confidence interval of the median (us)."""
    v = np.asarray(v, dtype=np.float64)
    rng = np.random.default_rng(seed)
    meds = np.median(v[rng.integers(0, len(v), size=(reps, len(v)))], axis=1)
    return (float(np.median(v)), float(np.percentile(meds, 2.5)),
            float(np.percentile(meds, 97.5)))


def _pick(stats, keys):
    """The key with the least median among keys."""
    return min(keys, key=lambda k: stats[k][0])


def _regret(stats, pick, best):
    return (stats[pick][0] - stats[best][0]) / stats[best][0]


def _agg(v):
    return {"mean": round(float(np.mean(v)), 4), "max": round(float(np.max(v)), 4)}


class SweepPoint:
    """A sweep workload on the device, its selector picks and its timings."""

    def __init__(self, name, B, torch):
        from workloads import sweep_workload
        self.name = name
        w = sweep_workload(name, with_tensors=False)
        self.w = w
        self.dw = DevWorkload(w, B, torch, synth_tensors=True)
        # the paper's column splits (owner-write), at the selector's pick
        self.params = B.launch_params(self.dw.wl)
        self.params_paper = B.launch_params(self.dw.wl)
        self.params_paper.c_min = 1
        self.pick = B.select_partition(self.dw.wl, self.params)[0]
        self.pick_paper = B.select_partition(self.dw.wl, self.params_paper)[0]
        wl_est, self._k = B.make_workload(w.T, w.H, w.I, w.E, w.topk, w.L, None)
        self.pick_est = B.select_partition(wl_est, B.launch_params(wl_est))[0]
        # token bands: (C, L) chosen together over L = 1..4
        self.params_bands = B.launch_params(self.dw.wl, 2)
        r, L, _ = B.select_partition_splits(self.dw.wl, self.params_bands, 1, 4)
        self.pick_bands = (r, 2, L)


def run_sweep(B, torch, samples, warmups, repeats=2, c_max=64):
    """The selector sweep: the 12 workloads x C = 0..c_max (owner-write,
    column splits, as the selector's launch uses), every C timed `samples`
    times (ABBA) after `warmups` passes; the whole sweep is repeated
    `repeats` times (independent passes, the second over the workloads in
    reverse order).  Regret = (t(pick) - t(best)) / t(best) on medians, for
    the library's candidate set 0..64 and for the paper's 1..64 (against
    the best in 1..64).  Also the token-band consumer over a grid of (C, L)
    with the selector's joint (C, L) pick."""
    from workloads import sweep_workloads
    names = [n for n, _ in sweep_workloads()]
    points = []
    for n in names:
        log(f"sweep setup {n}")
        points.append(SweepPoint(n, B, torch))
    Cs = list(range(0, c_max + 1))
    band_grid = [(c, 2, L) for L in (1, 2, 3, 4) for c in (0, 1, 2, 4, 8, 16, 24, 32, 48, 64)]
    runs = []     # per repeat: {name: {key: (median, lo, hi)}}
    for rep_i in range(repeats):
        order = points if rep_i % 2 == 0 else points[::-1]
        res = {}
        for pt in order:
            log(f"sweep {rep_i + 1}/{repeats} {pt.name}")
            # the band pick among its grid neighbours (ordered by L, then C),
            # not at an end of the pass
            band_keys = sorted(set(band_grid) | {pt.pick_bands}, key=lambda k: (k[2], k[0]))
            keys = Cs + band_keys
            t = time_configs(lambda c: launch_cfg(pt.dw, c), keys, samples, warmups, torch)
            assert pt.dw.ws.status() == 0
            res[pt.name] = {k: median_ci(v) for k, v in t.items()}
        runs.append(res)
    rows = []
    per_rep = {"regret": [], "paper": [], "estimate": [], "bands": []}
    for pt in points:
        row = {"w": pt.name, "r_expert": round(pt.w.r_expert, 2)}
        for ri, res in enumerate(runs):
            st = res[pt.name]
            best = _pick(st, Cs)
            best_dom = _pick(st, Cs[1:])
            keys_b = band_grid + [pt.pick_bands]
            best_b = _pick(st, keys_b)
            r = _regret(st, pt.pick, best)
            rp = _regret(st, pt.pick_paper, best_dom)
            re = _regret(st, pt.pick_est, best)
            rb = _regret(st, pt.pick_bands, best_b)
            per_rep["regret"].append((ri, r))
            per_rep["paper"].append((ri, rp))
            per_rep["estimate"].append((ri, re))
            per_rep["bands"].append((ri, rb))
            f = lambda k: [round(x, 1) for x in st[k]]   # noqa: E731
            row[f"s{ri + 1}"] = {
                "best": [best] + f(best), "pick": [pt.pick] + f(pt.pick), "regret": round(r, 4),
                "best_paper_set": [best_dom] + f(best_dom),
                "pick_paper": [pt.pick_paper] + f(pt.pick_paper), "regret_paper": round(rp, 4),
                "regret_estimate": round(re, 4),
                "bands_best": [best_b[0], best_b[2]] + f(best_b),
                "bands_pick": [pt.pick_bands[0], pt.pick_bands[2]] + f(pt.pick_bands),
                "regret_bands": round(rb, 4),
                "c0_vs_best_paper_set": round(st[0][0] / st[best_dom][0], 4)}
        rows.append(row)

    def by_rep(key):
        v = per_rep[key]
        reps = [_agg([r for i, r in v if i == k]) for k in range(repeats)]
        allv = [r for _, r in v]
        return {"mean": round(float(np.mean([x["mean"] for x in reps])), 4),
                "max": round(float(np.max(allv)), 4),
                "per_sweep_mean": [x["mean"] for x in reps],
                "per_sweep_max": [x["max"] for x in reps]}

    summary = {"workloads": len(rows), "samples_per_C": samples, "warmups": warmups,
               "sweeps": repeats, "C_range": [0, c_max],
               "regret": by_rep("regret"), "regret_paper_set": by_rep("paper"),
               "regret_estimate": by_rep("estimate"), "regret_bands": by_rep("bands")}
    detail = {"per_workload": rows,
              "us_by_C_sweep1": {pt.name: {str(c): round(runs[0][pt.name][c][0], 1) for c in Cs}
                                 for pt in points},
              "bands_us_by_C_L": [{pt.name: {f"C{k[0]}_L{k[2]}": round(res[pt.name][k][0], 1)
                                             for k in band_grid + [pt.pick_bands]}
                                   for pt in points} for res in runs]}
    return summary, detail, points, runs


def model_validation(B, torch, points, runs, Cs):
    """The makespan model against the measured sweep: T(C) in compute waves
    times the measured mean tile time (one traced launch at C = 0) against
    the measured median, per workload; and, on two workloads, the split
    arrival and finish times A_s, F_s rebuilt from the traced tile and task
    timestamps at C = 16 and C = 64 against the model's."""
    out = []
    for pt in points:
        dw = pt.dw
        _, tiles, _ = dw.trace(0)
        t_tile = float((tiles[:, 3] - tiles[:, 0]).mean()) * TICK_S * 1e6
        n, table, den = B.select_evaluate(dw.wl, pt.params)
        pred = {pt.params.c_min + i: table[i] / den * t_tile for i in range(n) if table[i] >= 0}
        meas = {c: runs[0][pt.name][c][0] for c in Cs}
        errs = {c: (pred[c] - meas[c]) / meas[c] for c in Cs if c in pred}
        dom = [c for c in Cs if c >= 1 and c in errs]
        rank_p = np.argsort(np.argsort([pred[c] for c in dom]))
        rank_m = np.argsort(np.argsort([meas[c] for c in dom]))
        rho_s = float(np.corrcoef(rank_p, rank_m)[0, 1])
        out.append({"w": pt.name, "tile_us": round(t_tile, 2),
                    "mape_paper_set": round(float(np.mean([abs(errs[c]) for c in dom])), 4),
                    "err_C0": round(errs[0], 4), "err_C16": round(errs[16], 4),
                    "err_C64": round(errs[64], 4), "spearman_paper_set": round(rho_s, 4),
                    "pred_over_meas_T0_T64": round((pred[0] / pred[64]) / (meas[0] / meas[64]), 4)})
    splits = []
    for pt in points:
        if pt.name not in ("sweep_T16384_uniform", "sweep_T32768_uniform"):
            continue
        dw = pt.dw
        part0 = B.select_partition(dw.wl, pt.params)[1]
        W_comp, W_comm = int(part0.W_comp), int(part0.W_comm)
        _, tiles0, _ = dw.trace(0)
        t_tile = float((tiles0[:, 3] - tiles0[:, 0]).mean()) * TICK_S * 1e6
        for C in (16, 64):
            _, tiles, tasks = dw.trace(C)
            t0 = tiles[:, 0].min()
            L = dw.w.L
            A = [float((tiles[s * W_comp:(s + 1) * W_comp, 3].max() - t0) * TICK_S * 1e6)
                 for s in range(L)]
            # (the last split's records run to the end: its tasks are finer)
            F = [float((tasks[s * W_comm:(s + 1) * W_comm if s < L - 1 else None, 2].max()
                        - t0) * TICK_S * 1e6) for s in range(L)]
            # the model's A_s and F_s of this candidate, as the library evaluates them
            _, _, den, A_m, F_m = B.select_candidate(dw.wl, pt.params, C)
            splits.append({"w": pt.name, "C": C,
                           "A_us_meas": [round(x, 1) for x in A],
                           "A_us_model": [round(a / den * t_tile, 1) for a in A_m],
                           "F_us_meas": [round(x, 1) for x in F],
                           "F_us_model": [round(f / den * t_tile, 1) for f in F_m]})
    return {"per_workload": out,
            "mape_paper_set_mean": round(float(np.mean([o["mape_paper_set"] for o in out])), 4),
            "err_C0_mean": round(float(np.mean([o["err_C0"] for o in out])), 4),
            "spearman_paper_set_mean": round(float(np.mean([o["spearman_paper_set"] for o in out])), 4),
            "split_times": splits}


def rho_validation(B, torch, reps=5, C_ref=32):
    """rho measured on each configuration by the calibration procedure (mean
    consumer-task time over mean compute-tile time in traced launches at
    C = 32) against the rho the selector would use (the library's, from
    moe_select_candidate): eq:rho-scaling from the calibration on the
    DeepSeek-V2-Lite-like share (with the task-token factor of the launch),
    and the same with the k/H-aware extension (rho_kh = 1)."""
    from workloads import config
    rows = []
    for name in ("tiny", "granite", "qwen", "dsv2lite"):
        w = config(name)
        dw = DevWorkload(w, B, torch)
        for _ in range(3):
            dw.run(C_ref)
        torch.cuda.synchronize()
        task_t, tile_t = [], []
        for _ in range(reps):
            _, tiles, tasks = dw.trace(C_ref)
            tile_t.append((tiles[:, 3] - tiles[:, 0]).mean())
            task_t.append(task_busy(dw, tasks).mean())
        tile_us = float(np.median(tile_t)) * TICK_S * 1e6
        task_us = float(np.median(task_t)) * TICK_S * 1e6
        p = B.launch_params(dw.wl)
        p.rho_kh = 0
        _, n0, d0, _, _ = B.select_candidate(dw.wl, p, 0)
        p.rho_kh = 1
        _, n1, d1, _, _ = B.select_candidate(dw.wl, p, 0)
        paper, kh = n0 / d0, n1 / d1
        meas = task_us / tile_us
        rows.append({"w": name, "I": w.I, "topk": w.topk, "task_tokens": p.comm_tile_m,
                     "tile_us": round(tile_us, 2), "task_us": round(task_us, 2),
                     "rho_measured": round(meas, 3), "rho_paper": round(float(paper), 3),
                     "rho_kh": round(float(kh), 3),
                     "err_paper": round(float(paper) / meas - 1, 3),
                     "err_kh": round(float(kh) / meas - 1, 3)})
        del dw
        torch.cuda.empty_cache()
    return rows


def saturation(B, torch, samples, warmups, name="sweep_T16384_uniform"):
    """The one-time saturation characterisation that sets C_max
    (eq:c-domain): C = 32..192 on a workload whose time still falls at
    C = 64; where does T(C) stop falling?"""
    pt = SweepPoint(name, B, torch)
    Cs = [32, 48, 56, 64, 72, 80, 96, 112, 128, 160, 192]
    t = time_configs(lambda c: pt.dw.run(c), Cs, samples, warmups, torch)
    st = {c: median_ci(v) for c, v in t.items()}
    best = _pick(st, Cs)
    return {"w": name, "us_by_C": {str(c): [round(x, 1) for x in st[c]] for c in Cs},
            "best_C": best, "best_us": round(st[best][0], 1)}


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
    settle_calls(list(fns.values()), torch, rounds=1)
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
    # the per-token brute force (one vector-matrix product per routed row)
    # on the tiny configuration, where it runs in full
    from workloads import config
    wt = config("tiny")
    t0 = time.perf_counter()
    oc.combine_bruteforce(wt.x_perm, wt.w2, wt.expert_offsets, wt.token_ids, wt.gate_w, wt.T)
    bf_s = time.perf_counter() - t0
    return {"value": round(flops / per / 1e12, 4), "unit": "TFLOP/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"whole {w.name} workload (numpy fp32 per-expert matmul + per-token "
                      f"weighted sum), {n} run(s), {per * 1e3:.1f} ms each; "
                      f"host os.cpu_count()={os.cpu_count()}",
            "bruteforce_tiny": {"seconds": round(bf_s, 3), "tokens": wt.T, "rows": wt.Mtot,
                                "tflops": round(2 * wt.Mtot * wt.I * wt.H / bf_s / 1e12, 5)}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="dsv2lite")
    ap.add_argument("--consumers", type=int, default=-1)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--sweep-samples", type=int, default=30,
                    help="timed samples per configuration in the selector sweep (ABBA)")
    ap.add_argument("--sweep-warmups", type=int, default=20,
                    help="untimed passes over all configurations before the samples")
    ap.add_argument("--sweep-repeats", type=int, default=2,
                    help="independent repetitions of the whole sweep")
    ap.add_argument("--no-validate", action="store_true",
                    help="skip the model-against-measurement validation and the C_max sweep")
    ap.add_argument("--detail-out", default="",
                    help="write the per-workload sweep tables (JSON) to this path")
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
        dw.run(32, mode=2)
        torch.cuda.synchronize()
        print(json.dumps({"calibration": calibrate(dw),
                          "calibration_scatter": calibrate(dw, mode=1),
                          "calibration_bands": calibrate(dw, mode=2),
                          "kernel_sha": kernel_sha()}), flush=True)
        return
    stream = torch.cuda.current_stream()

    # selector cost on the host (pure C++, no HIP calls), 10^5 calls through
    # ctypes; the same loop around a call that does nothing (the ABI version)
    # gives the ctypes overhead, which the net figure leaves out.  Measured
    # before the launches, so that no idle gap separates the warm-up from the
    # timed steps.
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

    log("settle")
    C_used = dw.run(args.consumers)
    settle_n = settle(dw, args.consumers, torch)
    log("warmup")
    for _ in range(args.warmup):
        dw.run(args.consumers)
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    log(f"timing {args.steps} steps, C={C_used}")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        starts[i].record(stream)
        dw.run(args.consumers)
        ends[i].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    st = dw.ws.status()
    assert st == 0, B.strerror(st)
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
        "settle_launches": settle_n,
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
        summary, detail, points, runs = run_sweep(B, torch, args.sweep_samples,
                                                  args.sweep_warmups, args.sweep_repeats)
        # short top-level keys first, so that a truncated line still has them
        head = {"sweep_regret": {k: summary["regret"][k] for k in ("mean", "max")},
                "sweep_regret_paper_set": {k: summary["regret_paper_set"][k]
                                           for k in ("mean", "max")},
                "sweep_regret_bands": {k: summary["regret_bands"][k] for k in ("mean", "max")}}
        res = {**{k: res[k] for k in list(res)[:13]}, **head,
               **{k: res[k] for k in list(res)[13:]}}
        res["sweep"] = summary
        if not args.no_validate:
            log("model against measurement")
            res["model_validation"] = model_validation(B, torch, points, runs,
                                                       list(range(0, 65)))
        del points
        torch.cuda.empty_cache()
        if not args.no_validate:
            log("C saturation")
            res["c_max_saturation"] = saturation(B, torch, args.sweep_samples,
                                                 args.sweep_warmups)
            log("rho across the configurations")
            res["rho_validation"] = rho_validation(B, torch)
        if args.detail_out:
            detail["model_validation"] = res.get("model_validation")
            with open(args.detail_out, "w") as f:
                json.dump(detail, f)
    if not args.no_cpu:
        log("timing the CPU oracle")
        res["cpu_baseline"] = cpu_baseline(w)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
