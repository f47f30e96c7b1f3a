"""GPU: moe_gemm2_combine_noalloc, the entry point for callers that cannot
allocate (its workspace is the library's own scratch), against
moe_gemm2_combine_ex with a caller workspace on the same inputs: two calls in
a row, the second with a smaller input, then the larger one again, in both
consumer modes.  Owner-write (mode 0) must match bitwise, the atomic scatter
(mode 1) to the parity bar; both also against the oracle."""
import numpy as np
import pytest

from oracle import combine as oc
from workloads import config, custom

pytestmark = pytest.mark.gpu


def _check(got, ref, what=""):
    rl2 = oc.rel_l2(got, ref)
    mab = oc.max_abs_ratio(got, ref)
    print(f"{what}: rel_l2={rl2:.3e} max_abs/max_ref={mab:.3e}", flush=True)
    assert np.isfinite(got).all()
    assert rl2 <= oc.REL_L2_TOL, (what, rl2)
    assert mab <= oc.MAX_ABS_TOL, (what, mab)


def _noalloc(w, dev, C, mode):
    import torch

    from paper_2609_07536_amd import binding as B
    x, w2, off, tid, g = dev
    out = torch.full((w.T, w.H), float("nan"), dtype=torch.float32, device="cuda")
    used = B.combine_noalloc(x, w2, off, tid, g, out, T=w.T, splits=w.L, topk=w.topk,
                             counts=w.counts, num_consumers=C, mode=mode)
    torch.cuda.synchronize()
    return out.cpu().numpy(), used


@pytest.mark.parametrize("mode", [0, 1])
def test_noalloc_matches_workspace_entry_point(gpu_lib, mode):
    import gpu_util
    big = config("granite")      # the largest configuration that fits the scratch
    small = custom(T=700, H=512, I=96, E=6, topk=3, L=2, routing=("zipf", 1.0), seed=51)
    cases = []
    for name, w in (("granite", big), ("small", small)):
        ref = oc.combine_reference(w.x_perm, w.w2, w.expert_offsets, w.token_ids, w.gate_w, w.T)
        dev = gpu_util.to_device(w)
        cases.append((name, w, ref, dev))
    for C in (-1, 0, 5):
        # the existing entry point with a caller workspace, on the same inputs
        want = {}
        for name, w, ref, dev in cases:
            print(f"combine_ex {name} mode={mode} C={C}", flush=True)
            got, used, _ = gpu_util.run(w, C=C, dev=dev, mode=mode)
            _check(got, ref, f"ex {name} mode={mode} C={used}")
            want[name] = (got, used)
        # the no-alloc entry point: larger, smaller, larger again, back to back
        for name, w, ref, dev in cases + cases[:1]:
            print(f"noalloc {name} mode={mode} C={C}", flush=True)
            got, used = _noalloc(w, dev, C, mode)
            assert used == want[name][1]
            _check(got, ref, f"noalloc {name} mode={mode} C={used}")
            if mode == 0:
                assert np.array_equal(got.view(np.uint32), want[name][0].view(np.uint32)), name
            else:
                _check(got, want[name][0], f"noalloc vs ex {name} C={used}")


def test_noalloc_rejects_workloads_beyond_the_scratch(gpu_lib):
    """A workload whose workspace exceeds the scratch is refused on the host,
    before anything is enqueued; the next call is unaffected."""
    import torch

    import gpu_util
    from paper_2609_07536_amd import binding as B
    w = config("qwen", with_tensors=False)
    wl, _ = B.make_workload(w.T, w.H, w.I, w.E, w.topk, w.L, rows=w.Mtot)
    assert B.workspace_size(wl) > B.NOALLOC_SCRATCH_BYTES
    x = torch.zeros((w.Mtot, w.I), dtype=torch.bfloat16, device="cuda")
    w2 = torch.zeros((w.E, w.I, w.H), dtype=torch.bfloat16, device="cuda")
    off = torch.from_numpy(w.expert_offsets).cuda()
    tid = torch.from_numpy(w.token_ids).cuda()
    g = torch.from_numpy(w.gate_w).cuda()
    out = torch.full((w.T, w.H), 5.0, dtype=torch.float32, device="cuda")
    with pytest.raises(B.MoeError) as ei:
        B.combine_noalloc(x, w2, off, tid, g, out, T=w.T, splits=w.L, topk=w.topk)
    assert ei.value.code == B.MOE_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert bool((out == 5.0).all())
    small = custom(T=300, H=256, I=32, E=3, topk=2, L=1, routing=("uniform",), seed=52)
    ref = oc.combine_reference(small.x_perm, small.w2, small.expert_offsets, small.token_ids,
                               small.gate_w, small.T)
    got, _ = _noalloc(small, gpu_util.to_device(small), -1, 0)
    _check(got, ref, "noalloc after a rejected call")
