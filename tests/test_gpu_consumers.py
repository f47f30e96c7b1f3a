"""GPU: the dedicated-consumer path (C >= 1, the paper's mechanism) at full
size, the readiness protocol under delayed publishes, 1000 back-to-back
launches on one workspace, and one workspace reused across layouts.

Owner-write sums each token's rows in ascending row order whatever the
partition, so its output is bitwise the same for every C (Method, "System
Integration and Correctness": only C and the reservation change); the
atomic scatter is compared with the oracle to the bar.
"""
import os

import numpy as np
import pytest

from oracle import combine as oc
from workloads import config, custom, sweep_workload

pytestmark = pytest.mark.gpu

_cache = {}


def _check(got, ref, what=""):
    rl2 = oc.rel_l2(got, ref)
    mab = oc.max_abs_ratio(got, ref)
    print(f"{what}: rel_l2={rl2:.3e} max_abs/max_ref={mab:.3e}", flush=True)
    assert np.isfinite(got).all()
    assert rl2 <= oc.REL_L2_TOL, (what, rl2)
    assert mab <= oc.MAX_ABS_TOL, (what, mab)


def _full(name):
    """Workload, oracle output, device tensors, workspace and the C = 0
    output (checked against the oracle once)."""
    if name not in _cache:
        import gpu_util
        w = sweep_workload(name) if name.startswith("sweep_") else config(name)
        print(f"{name}: T={w.T} rows={w.Mtot} r_expert={w.r_expert:.2f}", flush=True)
        ref = oc.combine_reference(w.x_perm, w.w2, w.expert_offsets, w.token_ids, w.gate_w, w.T)
        dev = gpu_util.to_device(w)
        base, _, ws = gpu_util.run(w, C=0, dev=dev)
        _check(base, ref, f"{name} C=0")
        _cache.clear()   # one full-size workload resident at a time
        _cache[name] = (w, ref, dev, ws, base)
    return _cache[name]


@pytest.mark.parametrize("name,C", [("dsv2lite", 1), ("dsv2lite", 32), ("dsv2lite", 57),
                                    ("dsv2lite", 64), ("sweep_T32768_uniform", 57),
                                    ("sweep_T32768_uniform", 64)])
def test_dedicated_consumers_full_size_bitwise(gpu_lib, name, C):
    """C dedicated consumers on the DeepSeek-V2-Lite-like share and on the
    largest sweep workload: bitwise equal to the oracle-checked C = 0
    output; at C = 64 (the pick of the paper's candidate set) also against
    the oracle directly."""
    import gpu_util
    w, ref, dev, ws, base = _full(name)
    print(f"{name}: C={C}", flush=True)
    got, used, _ = gpu_util.run(w, C=C, dev=dev, workspace=ws)
    assert used == C
    assert np.array_equal(got.view(np.uint32), base.view(np.uint32)), (name, C)
    if C == 64:
        _check(got, ref, f"{name} C=64 vs oracle")


@pytest.mark.parametrize("mode,C", [(0, 56), (0, 60), (2, 0), (2, 1), (2, 8), (1, 0)])
def test_rotated_rounds_largest_sweep_shape(gpu_lib, mode, C):
    """T = 32768 has about 25 compute rounds, so workgroups whose P is a
    multiple of the n-tiles per m-tile take their tiles rotated by one more
    each round (C = 0, 56 and 60 with column splits, C = 0 and 8 with token
    bands; C = 1 with bands and C = 57 keep the plain order).  Owner-write
    results stay bitwise equal to the oracle-checked C = 0 output; the atomic
    scatter is checked against the oracle."""
    import gpu_util
    w, ref, dev, ws, base = _full("sweep_T32768_uniform")
    print(f"T=32768 mode={mode} C={C}", flush=True)
    got, used, _ = gpu_util.run(w, C=C, dev=dev, workspace=ws, mode=mode)
    assert used == C
    if mode == 1:
        _check(got, ref, f"T=32768 scatter C={C}")
    else:
        assert np.array_equal(got.view(np.uint32), base.view(np.uint32)), (mode, C)


def _mid(seed=21):
    return custom(T=2048, H=1024, I=256, E=16, topk=4, L=2, routing=("zipf", 1.0), seed=seed)


@pytest.mark.parametrize("C", [1, 64, 0])
def test_delayed_publishes(gpu_lib, C):
    """Every fourth compute workgroup holds each of its split publishes back
    by 200 us (a bounded spin, set from the host): consumers reach the
    split's flags long before they are all set, and the output is still
    bitwise the undelayed one."""
    import gpu_util
    w = _mid()
    ref = oc.combine_reference(w.x_perm, w.w2, w.expert_offsets, w.token_ids, w.gate_w, w.T)
    dev = gpu_util.to_device(w)
    base, _, ws = gpu_util.run(w, C=C, dev=dev)
    _check(base, ref, f"undelayed C={C}")
    old = os.environ.get("MOE_GEMM2_DEBUG_PUBLISH_DELAY")
    os.environ["MOE_GEMM2_DEBUG_PUBLISH_DELAY"] = "4:20000"
    try:
        for i in range(3):
            print(f"delayed publishes C={C} launch {i}", flush=True)
            got, used, ws = gpu_util.run(w, C=C, dev=dev, workspace=ws)
            assert np.array_equal(got.view(np.uint32), base.view(np.uint32)), (C, i)
        got, used, ws = gpu_util.run(w, C=C, dev=dev, workspace=ws, mode=1)
        _check(got, ref, f"delayed publishes scatter C={C}")
    finally:
        if old is None:
            del os.environ["MOE_GEMM2_DEBUG_PUBLISH_DELAY"]
        else:
            os.environ["MOE_GEMM2_DEBUG_PUBLISH_DELAY"] = old


def test_thousand_launches_one_workspace(gpu_lib):
    """1000 launches back to back on one workspace, cycling C over
    {0, 1, 8, 64} and both consumer modes: every owner-write output is
    bitwise the first one, every scatter output within the bar of it
    (compared on the device); stops at the first mismatch or error."""
    import torch

    import gpu_util
    from paper_2609_07536_amd import binding as B
    w = _mid(seed=22)
    ref = oc.combine_reference(w.x_perm, w.w2, w.expert_offsets, w.token_ids, w.gate_w, w.T)
    x, w2, off, tid, g = gpu_util.to_device(w)
    wl, _ = B.make_workload(w.T, w.H, w.I, w.E, w.topk, w.L, w.counts)
    ws = B.Workspace(B.workspace_size(wl))
    out = torch.empty((w.T, w.H), dtype=torch.float32, device="cuda")
    B.combine(x, w2, off, tid, g, T=w.T, splits=w.L, topk=w.topk, counts=w.counts,
              num_consumers=8, out=out, workspace=ws)
    torch.cuda.synchronize()
    first = out.clone()
    _check(first.cpu().numpy(), ref, "first launch")
    ref_max = float(first.abs().max())
    plan = [(C, mode) for mode in (0, 1) for C in (0, 1, 8, 64)]
    for i in range(1000):
        C, mode = plan[i % len(plan)]
        out.fill_(float("nan"))
        B.combine(x, w2, off, tid, g, T=w.T, splits=w.L, topk=w.topk, counts=w.counts,
                  num_consumers=C, out=out, workspace=ws, mode=mode)
        if mode == 0:
            ok = bool(torch.equal(out, first))
        else:
            d = (out - first).abs().max()
            ok = bool(torch.isfinite(out).all()) and float(d) <= oc.MAX_ABS_TOL * ref_max
        if not ok or i % 100 == 99:
            st = ws.status()
            print(f"launch {i}: C={C} mode={mode} ok={ok} status={st}", flush=True)
            assert st == 0, B.strerror(st)
        assert ok, (i, C, mode)


def test_workspace_reused_across_layouts(gpu_lib):
    """One workspace (sized for the largest) used for workloads of different
    layouts in turn, larger and smaller, without re-initialising it in
    between: every output is right."""
    import gpu_util
    from paper_2609_07536_amd import binding as B
    shapes = [custom(T=3000, H=1024, I=128, E=12, topk=4, L=2, routing=("zipf", 1.0), seed=41),
              custom(T=700, H=512, I=96, E=6, topk=3, L=2, routing=("uniform",), seed=42),
              custom(T=5000, H=2048, I=64, E=40, topk=6, L=2, routing=("zipf", 0.8), seed=43),
              custom(T=300, H=256, I=32, E=3, topk=2, L=1, routing=("uniform",), seed=44)]
    need = 0
    for w in shapes:
        wl, _ = B.make_workload(w.T, w.H, w.I, w.E, w.topk, w.L)
        need = max(need, B.workspace_size(wl))
    ws = B.Workspace(need)
    refs = [oc.combine_reference(w.x_perm, w.w2, w.expert_offsets, w.token_ids, w.gate_w, w.T)
            for w in shapes]
    for rnd in range(2):
        for i, (w, ref) in enumerate(zip(shapes, refs)):
            for C, mode in ((0, 0), (5, 0), (0, 1)):
                print(f"relayout round {rnd} shape {i} C={C} mode={mode}", flush=True)
                got, used, ws = gpu_util.run(w, C=C, workspace=ws, mode=mode)
                _check(got, ref, f"shape {i} C={C} mode={mode}")


def test_fresh_workspaces_read_published_y_only(gpu_lib):
    """Regression for the readiness publish: a compute workgroup's release
    writes back the L2 and must wait for that write-back before it stores
    the flags, or a consumer on another XCD may read Y before it arrives.
    With a fresh (zeroed) workspace per launch such a read returns the
    workspace's zeros instead of the previous launch's identical Y, so the
    output differs.  Shapes whose tiles are a single reduction stage (I = 40)
    or have a partial width (H = 200) publish soonest after their stores;
    every launch must be bitwise equal to the first (mode 0 and token bands,
    dedicated consumers and the role switch)."""
    import gpu_util
    cases = [
        (custom(T=257, H=264, I=40, E=5, topk=2, L=1, routing=("uniform",), seed=13),
         [(0, None, None), (3, None, None)], 150),
        (custom(T=129, H=200, I=72, E=4, topk=2, L=1, routing=("zipf", 1.0), seed=13),
         [(5, 2, 5), (0, 2, 5)], 100),
    ]
    for w, cfgs, reps in cases:
        ref = oc.combine_reference(w.x_perm, w.w2, w.expert_offsets, w.token_ids, w.gate_w, w.T)
        dev = gpu_util.to_device(w)
        base, _, _ = gpu_util.run(w, C=0, dev=dev)
        _check(base, ref, f"fresh T={w.T} H={w.H} I={w.I} base")
        for C, mode, L in cfgs:
            print(f"fresh workspaces T={w.T} H={w.H} I={w.I} C={C} mode={mode} L={L} x{reps}",
                  flush=True)
            for it in range(reps):
                got, _, _ = gpu_util.run(w, C=C, dev=dev, mode=mode, splits=L)
                assert np.array_equal(got.view(np.uint32), base.view(np.uint32)), (C, mode, L, it)
