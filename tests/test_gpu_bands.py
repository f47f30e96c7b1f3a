"""GPU parity of the token-band consumer (moe_gemm2_combine_ex mode 2):
pipeline splits along the routed rows, each task waiting for the bands that
hold its rows, agent-coherent reads of Y, compute workgroups draining into
consumers.  The owner-write sum order (ascending row per token) does not
depend on the split or the partition, so the output must be bitwise the
column-split owner-write output (mode 0) for every band count and C, and
within the bar of the oracle.
"""
import numpy as np
import pytest

from oracle import combine as oc
from workloads import config, custom, explicit

pytestmark = pytest.mark.gpu

_cache = {}


def _check(got, ref, what=""):
    rl2 = oc.rel_l2(got, ref)
    mab = oc.max_abs_ratio(got, ref)
    print(f"{what}: rel_l2={rl2:.3e} max_abs/max_ref={mab:.3e}", flush=True)
    assert np.isfinite(got).all()
    assert rl2 <= oc.REL_L2_TOL, (what, rl2)
    assert mab <= oc.MAX_ABS_TOL, (what, mab)


def _base(name):
    if name not in _cache:
        import gpu_util
        w = config(name)
        print(f"{name}: T={w.T} rows={w.Mtot}", flush=True)
        ref = oc.combine_reference(w.x_perm, w.w2, w.expert_offsets, w.token_ids, w.gate_w, w.T)
        dev = gpu_util.to_device(w)
        base, _, ws = gpu_util.run(w, C=0, dev=dev)
        _check(base, ref, f"{name} mode 0")
        _cache.clear()
        _cache[name] = (w, ref, dev, ws, base)
    return _cache[name]


@pytest.mark.parametrize("name", ["tiny", "granite", "qwen", "dsv2lite"])
@pytest.mark.parametrize("L", [1, 2, 4, 8])
def test_bands_configs_bitwise(gpu_lib, name, L):
    import gpu_util
    w, ref, dev, ws, base = _base(name)
    for C in (0, 1, 16, 48):
        print(f"{name} bands L={L} C={C}", flush=True)
        got, used, _ = gpu_util.run(w, C=C, dev=dev, workspace=ws, mode=2, splits=L)
        assert used == C
        if not np.array_equal(got.view(np.uint32), base.view(np.uint32)):
            _check(got, ref, f"{name} bands L={L} C={C}")
            raise AssertionError(f"{name} L={L} C={C}: not bitwise equal to mode 0")


EDGE = [
    ("ragged_small", 37, 64, 24, 3, 2, 1, ("uniform",)),
    ("one_expert", 300, 256, 64, 1, 1, 3, ("uniform",)),
    ("top1", 500, 512, 128, 8, 1, 2, ("zipf", 1.5)),
    ("k_tail_I40", 257, 264, 40, 5, 2, 4, ("uniform",)),
    ("H_not_tile", 129, 200, 72, 4, 2, 5, ("zipf", 1.0)),
    ("wide_H", 300, 4096, 64, 4, 2, 2, ("uniform",)),
    ("many_experts", 1000, 256, 64, 200, 8, 8, ("zipf", 0.5)),
    ("topk_16", 200, 128, 32, 20, 16, 16, ("uniform",)),
    ("single_token", 1, 1024, 512, 8, 2, 4, ("uniform",)),
    ("bands_past_tiles", 90, 512, 64, 6, 2, 16, ("zipf", 1.2)),
]


@pytest.mark.parametrize("case", EDGE, ids=[c[0] for c in EDGE])
def test_bands_edge_shapes(gpu_lib, case):
    """Ragged shapes; more bands than some experts have m-tiles (empty runs)."""
    import gpu_util
    name, T, H, I, E, k, L, routing = case
    w = custom(T=T, H=H, I=I, E=E, topk=k, L=1, routing=routing, seed=13)
    ref = oc.combine_reference(w.x_perm, w.w2, w.expert_offsets, w.token_ids, w.gate_w, w.T)
    dev = gpu_util.to_device(w)
    base, _, _ = gpu_util.run(w, C=0, dev=dev)
    _check(base, ref, f"{name} mode 0")
    for C in (0, 1, 5):
        got, used, _ = gpu_util.run(w, C=C, dev=dev, mode=2, splits=L)
        assert np.array_equal(got.view(np.uint32), base.view(np.uint32)), (name, C)


def test_bands_unsorted_rows(gpu_lib):
    """Rows inside each expert in a shuffled token order: bands then no
    longer follow token ranges, and the per-task band requirement (taken
    from the rows themselves) still gives the exact result."""
    import gpu_util
    w = custom(T=3000, H=1024, I=128, E=12, topk=4, L=1, routing=("zipf", 1.0), seed=14)
    rng = np.random.default_rng(7)
    perm = np.arange(w.Mtot)
    for e in range(w.E):
        a, b = int(w.expert_offsets[e]), int(w.expert_offsets[e + 1])
        perm[a:b] = a + rng.permutation(b - a)
    w.x_perm, w.token_ids, w.gate_w = w.x_perm[perm], w.token_ids[perm], w.gate_w[perm]
    ref = oc.combine_reference(w.x_perm, w.w2, w.expert_offsets, w.token_ids, w.gate_w, w.T)
    dev = gpu_util.to_device(w)
    base, _, _ = gpu_util.run(w, C=0, dev=dev)
    _check(base, ref, "unsorted mode 0")
    for L, C in ((4, 0), (4, 8), (8, 3)):
        got, used, _ = gpu_util.run(w, C=C, dev=dev, mode=2, splits=L)
        assert np.array_equal(got.view(np.uint32), base.view(np.uint32)), (L, C)


def test_bands_dropped_slots_and_no_rows(gpu_lib):
    import gpu_util
    rng = np.random.default_rng(5)
    T, H, I, E, k = 300, 512, 64, 6, 4
    sel, gates = [], []
    for t in range(T):
        n = int(rng.integers(0, k + 1))
        es = rng.choice([0, 2, 3, 5], size=min(n, 4), replace=False)
        sel.append(list(es))
        gates.append(list(rng.random(len(es)).astype(np.float32)))
    w = explicit(T, H, I, E, sel, gates)
    w.topk = k
    ref = oc.combine_reference(w.x_perm, w.w2, w.expert_offsets, w.token_ids, w.gate_w, w.T)
    empty = [t for t in range(T) if len(sel[t]) == 0]
    for L, C in ((1, 0), (3, 2), (6, 0)):
        got, used, _ = gpu_util.run(w, C=C, mode=2, splits=L)
        _check(got, ref, f"dropped bands L={L} C={C}")
        assert np.all(got[empty] == 0)
    w0 = explicit(50, 256, 32, 4, [[] for _ in range(50)], [[] for _ in range(50)])
    w0.topk = 2
    w0.x_perm = np.zeros((1, 32), dtype=np.uint16)
    w0.token_ids = np.zeros(1, dtype=np.int32)
    w0.gate_w = np.zeros(1, dtype=np.float32)
    got, used, _ = gpu_util.run(w0, C=2, counts=False, mode=2, splits=3)
    assert np.all(got == 0)


@pytest.mark.parametrize("name", ["sweep_T4096_zipf1.2", "sweep_T16384_uniform"])
def test_bands_selector_pick_bitwise(gpu_lib, name):
    """The token-band selector's joint (C, L) pick, the configuration the
    benchmark times (odd C such as 13 or 29 included), and the launch's own
    selection at that L (num_consumers = -1): bitwise the column-split
    owner-write output, which is checked against the oracle."""
    import gpu_util
    from paper_2609_07536_amd import binding as B
    from workloads import sweep_workload
    w = sweep_workload(name)
    print(f"{name}: T={w.T} rows={w.Mtot}", flush=True)
    ref = oc.combine_reference(w.x_perm, w.w2, w.expert_offsets, w.token_ids, w.gate_w, w.T)
    dev = gpu_util.to_device(w)
    sizes = [B.workspace_size(B.make_workload(w.T, w.H, w.I, w.E, w.topk, L, w.counts,
                                              rows=w.Mtot)[0]) for L in (1, 2, 3, 4)]
    ws = B.Workspace(max(sizes))
    base, _, _ = gpu_util.run(w, C=0, dev=dev, workspace=ws)
    _check(base, ref, f"{name} mode 0")
    wl1, _ = B.make_workload(w.T, w.H, w.I, w.E, w.topk, 1, w.counts, rows=w.Mtot)
    C, L, part = B.select_partition_splits(wl1, B.launch_params(wl1, 2), 1, 4)
    assert C >= 0 and 1 <= L <= 4
    for c in (C, -1):
        print(f"{name} bands pick C={C} L={L} (num_consumers {c})", flush=True)
        got, used, _ = gpu_util.run(w, C=c, dev=dev, workspace=ws, mode=2, splits=L)
        if c >= 0:
            assert used == C
        if not np.array_equal(got.view(np.uint32), base.view(np.uint32)):
            _check(got, ref, f"{name} bands C={used} L={L}")
            raise AssertionError(f"{name} bands C={used} L={L}: not bitwise equal to mode 0")
