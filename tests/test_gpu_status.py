"""GPU: the traced entry point, the device status word (bad routing, the
consumer watchdog) and recovery after an error.

Every failure here is forced from the host (bad ids in the routing arrays,
a tiny spin limit on the kernel's own bounded waits); every launch still
ends normally."""
import os

import numpy as np
import pytest

from oracle import combine as oc
from workloads import custom

pytestmark = pytest.mark.gpu


def _check(got, ref, what=""):
    rl2 = oc.rel_l2(got, ref)
    mab = oc.max_abs_ratio(got, ref)
    print(f"{what}: rel_l2={rl2:.3e} max_abs/max_ref={mab:.3e}", flush=True)
    assert np.isfinite(got).all()
    assert rl2 <= oc.REL_L2_TOL, (what, rl2)
    assert mab <= oc.MAX_ABS_TOL, (what, mab)


def _small(seed=5):
    return custom(T=700, H=512, I=96, E=6, topk=3, L=2, routing=("zipf", 1.0), seed=seed)


def _owner_tasks(w, p):
    """Owner-write task records of a launch: tasks_per_split for every split
    but the last, whose tasks hold comm_tile_m_last tokens."""
    tm, tm_last = p.comm_tile_m, p.comm_tile_m_last or p.comm_tile_m
    cb = (w.H // w.L + 1023) // 1024
    return (w.L - 1) * -(-w.T // tm) * cb + -(-w.T // tm_last) * cb


@pytest.mark.parametrize("T", [700, 8192])
def test_traced_matches_untraced(gpu_lib, T):
    """(T = 8192 has 32-token tasks and a last split of 16-token ones.)"""
    import torch

    import gpu_util
    from paper_2609_07536_amd import binding as B
    w = custom(T=T, H=512, I=96, E=6, topk=3, L=2, routing=("zipf", 1.0), seed=5)
    dev = gpu_util.to_device(w)
    for C in (0, 4):
        plain, used, ws = gpu_util.run(w, C=C, dev=dev)
        wl, _ = B.make_workload(w.T, w.H, w.I, w.E, w.topk, w.L, w.counts)
        trace = torch.zeros(B.trace_size(wl) // 8, dtype=torch.int64, device="cuda")
        traced, used2, _ = gpu_util.run(w, C=C, dev=dev, workspace=ws, trace=trace)
        assert used2 == used
        assert np.array_equal(traced.view(np.uint32), plain.view(np.uint32))
        tr = trace.cpu().numpy().astype(np.int64)
        p = B.launch_params(wl)
        r, part = B.select_partition(wl, p)
        n_tiles = int(part.W_comp) * w.L
        t = tr[:4 * n_tiles].reshape(-1, 4)
        assert (t[:, 3] > 0).all(), "every tile publishes"
        assert (np.diff(t, axis=1) >= 0).all(), "tile timestamps ordered"
        n_tasks = _owner_tasks(w, p)
        if T == 8192:
            assert (p.comm_tile_m, p.comm_tile_m_last) == (32, 16)
        rows = w.x_perm.shape[0]
        max_tiles = w.L * (-(-(w.H // w.L) // 256)) * (-(-rows // 256) + w.E)
        k = tr[4 * max_tiles:4 * max_tiles + 4 * n_tasks].reshape(-1, 4)
        assert (k[:, 2] > 0).all(), "every consumer task recorded"
        assert (k[:, 1] >= k[:, 0]).all() and (k[:, 2] >= k[:, 1]).all()
        assert (k[:, 3] >= 0).all() and (k[:, 3] < 4096).all()   # block ids


def test_bad_token_ids_flagged_and_skipped(gpu_lib):
    import gpu_util
    from paper_2609_07536_amd import binding as B
    w = _small(seed=6)
    rng = np.random.default_rng(1)
    bad = rng.choice(w.token_ids.size, size=9, replace=False)
    gate_ref = w.gate_w.copy()
    gate_ref[bad] = 0.0                        # a skipped row contributes nothing
    ref = oc.combine_reference(w.x_perm, w.w2, w.expert_offsets, w.token_ids, gate_ref, w.T)
    w.token_ids = w.token_ids.copy()
    w.token_ids[bad[:5]] = w.T + 7             # past the last token
    w.token_ids[bad[5:]] = -3                  # negative
    for C in (0, 3):
        got, used, ws = gpu_util.run(w, C=C, check_status=False)
        assert ws.status() == B.MOE_ERR_BAD_ROUTING
        assert ws.status(clear=True) == B.MOE_ERR_BAD_ROUTING
        assert ws.status() == 0                # cleared
        _check(got, ref, f"bad ids C={used}")


def test_token_with_too_many_rows_flagged(gpu_lib):
    import gpu_util
    from paper_2609_07536_amd import binding as B
    w = _small(seed=7)
    # give token 0 one row more than top-k (taken from some other token)
    rows0 = np.flatnonzero(w.token_ids == 0)
    assert rows0.size == w.topk
    donor_row = int(np.flatnonzero(w.token_ids != 0)[0])
    donor = int(w.token_ids[donor_row])
    ref = oc.combine_reference(w.x_perm, w.w2, w.expert_offsets, w.token_ids, w.gate_w, w.T)
    w.token_ids = w.token_ids.copy()
    w.token_ids[donor_row] = 0
    got, used, ws = gpu_util.run(w, C=2, check_status=False)
    assert ws.status(clear=True) == B.MOE_ERR_BAD_ROUTING
    keep = np.ones(w.T, dtype=bool)
    keep[[0, donor]] = False                   # which of token 0's rows is dropped is unordered
    _check(got[keep], ref[keep], "too many rows")
    assert np.isfinite(got).all()


def test_bad_expert_offsets_clamped(gpu_lib):
    import gpu_util
    from paper_2609_07536_amd import binding as B
    w = _small(seed=8)
    off = w.expert_offsets.copy()
    off[2], off[3] = off[3] + 5, off[2]        # decreasing, and past its neighbour
    off[-1] = off[-1] + 1000                   # past the rows (clamped to rows)
    w.expert_offsets = off
    got, used, ws = gpu_util.run(w, C=0, counts=False, check_status=False)
    assert ws.status(clear=True) == B.MOE_ERR_BAD_ROUTING
    assert np.isfinite(got).all()


def test_watchdog_expires_and_next_launch_is_clean(gpu_lib):
    """A spin limit of 1 makes every consumer wait give up at once: the
    launch ends with MOE_ERR_TIMEOUT; the next launch on the same workspace
    is correct."""
    import gpu_util
    from paper_2609_07536_amd import binding as B
    w = _small(seed=9)
    ref = oc.combine_reference(w.x_perm, w.w2, w.expert_offsets, w.token_ids, w.gate_w, w.T)
    dev = gpu_util.to_device(w)
    old = os.environ.get("MOE_GEMM2_SPIN_LIMIT")
    os.environ["MOE_GEMM2_SPIN_LIMIT"] = "1"
    try:
        _, used, ws = gpu_util.run(w, C=8, dev=dev, check_status=False)
        st = ws.status(clear=True)
    finally:
        if old is None:
            del os.environ["MOE_GEMM2_SPIN_LIMIT"]
        else:
            os.environ["MOE_GEMM2_SPIN_LIMIT"] = old
    assert st == B.MOE_ERR_TIMEOUT, B.strerror(st)
    got, used, ws = gpu_util.run(w, C=8, dev=dev, workspace=ws)
    _check(got, ref, "after timeout")


def test_two_streams_at_once(gpu_lib):
    """Two launches in flight together on two streams with two workspaces
    (each with its own consumers or the role switch) both come out right.
    The launches share no device state, and a grid that is not fully
    resident still drains: compute workgroups never wait while they hold
    tiles, and with C = 0 a workgroup serves (and waits for) consumer tasks
    only once every workgroup of its grid has started."""
    import torch

    import gpu_util
    from paper_2609_07536_amd import binding as B
    wa = _small(seed=11)
    wb = custom(T=1500, H=1024, I=128, E=12, topk=4, L=2, routing=("zipf", 0.8), seed=12)
    refs = [oc.combine_reference(w.x_perm, w.w2, w.expert_offsets, w.token_ids, w.gate_w, w.T)
            for w in (wa, wb)]
    devs = [gpu_util.to_device(w) for w in (wa, wb)]
    outs = [torch.empty((w.T, w.H), dtype=torch.float32, device="cuda") for w in (wa, wb)]
    wss = []
    for w in (wa, wb):
        wl, _ = B.make_workload(w.T, w.H, w.I, w.E, w.topk, w.L, w.counts)
        wss.append(B.Workspace(B.workspace_size(wl)))
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]   # default priority
    for Cs in ((0, 4), (8, 0), (3, 3)):
        for w, d, o, ws, st, C in zip((wa, wb), devs, outs, wss, streams, Cs):
            x, w2, off, tid, g = d
            B.combine(x, w2, off, tid, g, T=w.T, splits=w.L, topk=w.topk, counts=w.counts,
                      num_consumers=C, out=o, workspace=ws, stream=st)
        torch.cuda.synchronize()
        for w, o, ws, ref, C in zip((wa, wb), outs, wss, refs, Cs):
            assert ws.status() == 0
            _check(o.cpu().numpy(), ref, f"two streams C={C}")


def test_scatter_bad_token_ids_flagged_and_skipped(gpu_lib):
    import gpu_util
    from paper_2609_07536_amd import binding as B
    w = _small(seed=16)
    rng = np.random.default_rng(2)
    bad = rng.choice(w.token_ids.size, size=9, replace=False)
    gate_ref = w.gate_w.copy()
    gate_ref[bad] = 0.0
    ref = oc.combine_reference(w.x_perm, w.w2, w.expert_offsets, w.token_ids, gate_ref, w.T)
    w.token_ids = w.token_ids.copy()
    w.token_ids[bad[:5]] = w.T
    w.token_ids[bad[5:]] = -1
    for C in (0, 3):
        got, used, ws = gpu_util.run(w, C=C, check_status=False, mode=1)
        assert ws.status(clear=True) == B.MOE_ERR_BAD_ROUTING
        _check(got, ref, f"scatter bad ids C={used}")


def test_scatter_traced_records_every_tile_task(gpu_lib):
    import torch

    import gpu_util
    from paper_2609_07536_amd import binding as B
    w = _small(seed=17)
    ref = oc.combine_reference(w.x_perm, w.w2, w.expert_offsets, w.token_ids, w.gate_w, w.T)
    wl, _ = B.make_workload(w.T, w.H, w.I, w.E, w.topk, w.L, w.counts)
    r, part = B.select_partition(wl, B.default_params(0))
    n_tiles = int(part.W_comp) * w.L
    for C in (0, 4):
        trace = torch.zeros(B.trace_size(wl) // 8, dtype=torch.int64, device="cuda")
        got, used, _ = gpu_util.run(w, C=C, trace=trace, mode=1)
        _check(got, ref, f"scatter traced C={used}")
        tr = trace.cpu().numpy().astype(np.int64)
        rows = w.x_perm.shape[0]
        max_tiles = w.L * (-(-(w.H // w.L) // 256)) * (-(-rows // 256) + w.E)
        owner_tasks = _owner_tasks(w, B.launch_params(wl))
        assert len(tr) == 4 * max_tiles + 4 * max(owner_tasks, max_tiles)
        t = tr[:4 * n_tiles].reshape(-1, 4)
        assert (t[:, 3] > 0).all()
        k = tr[4 * max_tiles:4 * max_tiles + 4 * n_tiles].reshape(-1, 4)
        assert (k[:, 2] > 0).all(), "every tile scattered once"
        assert (k[:, 1] >= k[:, 0]).all() and (k[:, 2] >= k[:, 1]).all()
        assert (tr[4 * max_tiles + 4 * n_tiles:] == 0).all()



def test_graph_capture_replays(gpu_lib):
    """The stage captured in a HIP graph (host counts absent, so the selector
    uses the even-load estimate and needs nothing from the device) and
    replayed: every replay equals the eager launch bitwise, with eager
    launches and synchronisations between replays.  Each launch's epoch
    comes from the workspace, so replays of the same captured arguments
    never see the previous replay's flags."""
    import torch

    import gpu_util
    from paper_2609_07536_amd import binding as B
    w = custom(T=1200, H=1024, I=128, E=12, topk=4, L=2, routing=("zipf", 1.0), seed=31)
    ref = oc.combine_reference(w.x_perm, w.w2, w.expert_offsets, w.token_ids, w.gate_w, w.T)
    x, w2, off, tid, g = gpu_util.to_device(w)
    wl, _ = B.make_workload(w.T, w.H, w.I, w.E, w.topk, w.L)
    B.default_params(0)                       # device facts cached before the capture
    for mode in (0, 1):
        ws = B.Workspace(B.workspace_size(wl))
        out = torch.empty((w.T, w.H), dtype=torch.float32, device="cuda")
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):         # warm-up launch on the capture stream
            B.combine(x, w2, off, tid, g, T=w.T, splits=w.L, topk=w.topk, out=out,
                      workspace=ws, stream=side, mode=mode)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        eager = out.cpu().numpy().copy()
        _check(eager, ref, f"graph eager mode={mode}")
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=side):
            B.combine(x, w2, off, tid, g, T=w.T, splits=w.L, topk=w.topk, out=out,
                      workspace=ws, stream=side, mode=mode)
        for i in range(4):
            out.fill_(float("nan"))
            graph.replay()
            torch.cuda.synchronize()
            got = out.cpu().numpy()
            if mode == 0:
                assert np.array_equal(got.view(np.uint32), eager.view(np.uint32)), i
            else:
                _check(got, ref, f"graph replay {i} scatter")
            # an eager launch on the same workspace between replays
            B.combine(x, w2, off, tid, g, T=w.T, splits=w.L, topk=w.topk, out=out,
                      workspace=ws, mode=mode)
            torch.cuda.synchronize()
            assert ws.status() == 0
