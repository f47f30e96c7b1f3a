"""GPU parity of the up-projection (moe_gemm1_swiglu) and of the whole
post-router layer (moe_layer_forward) against the CPU oracle, through the C
ABI.

x_perm is bf16: the GPU and the oracle round nearly equal fp32 values, whose
summation orders differ, so an element may differ by one bf16 unit in the
last place where its fp32 value lies at a rounding midpoint; the test
demands at most one such unit everywhere and bit equality almost everywhere.
The layer's output meets the stage's bar (rel-L2 <= 5e-3, max-abs <= 1e-2
max|ref|)."""
import numpy as np
import pytest

from oracle import combine as oc
from oracle import layer as ol
from workloads import config, custom, explicit, layer_inputs

pytestmark = pytest.mark.gpu


def _dev(w, hidden, w1):
    import torch
    from paper_2609_07536_amd import binding as B
    d = "cuda"
    h = torch.from_numpy(hidden.view(np.int16)).to(d).view(torch.bfloat16)
    w1g = torch.from_numpy(w1.view(np.int16)).to(d).view(torch.bfloat16)
    w1p = B.pack_w1(w1g)
    w2 = torch.from_numpy(w.w2.view(np.int16)).to(d).view(torch.bfloat16)
    off = torch.from_numpy(w.expert_offsets.astype(np.int32)).to(d)
    tid = torch.from_numpy(w.token_ids.astype(np.int32)).to(d)
    g = torch.from_numpy(w.gate_w.astype(np.float32)).to(d)
    return h, w1g, w1p, w2, off, tid, g


def _x_check(got_bits, act, ref_bits, what):
    """x_perm against the oracle: bit-equal almost everywhere, and within
    one bf16 rounding (2^-8 relative) of the oracle's fp32 activation plus a
    small absolute slack for outputs near zero, where a dot product's
    cancellation makes fp32 summation-order differences relatively large."""
    got = oc.bf16_bits_to_f32(got_bits)
    frac_equal = float(np.mean(got_bits == ref_bits)) if got_bits.size else 1.0
    scale = float(np.max(np.abs(act))) if act.size else 0.0
    err = np.abs(got.astype(np.float64) - act)
    bound = 2.0 ** -8 * np.abs(act) + 1e-5 * scale
    print(f"{what}: bit-equal {frac_equal:.5f}, max err/bound {np.max(err / bound) if act.size else 0:.3f}",
          flush=True)
    assert np.all(err <= bound), what
    assert frac_equal >= 0.99, what


def _check_bar(got, ref, what):
    rl2, mab = oc.rel_l2(got, ref), oc.max_abs_ratio(got, ref)
    print(f"{what}: rel_l2={rl2:.3e} max_abs/max_ref={mab:.3e}", flush=True)
    assert np.isfinite(got).all()
    assert rl2 <= oc.REL_L2_TOL and mab <= oc.MAX_ABS_TOL, what


def test_pack_w1_layout(gpu_lib):
    """The packed layout as documented: column 32b + j is gate column 16b + j,
    column 32b + 16 + j is up column 16b + j."""
    import torch
    from paper_2609_07536_amd import binding as B
    E, H, I = 3, 5, 48
    src = np.random.default_rng(0).integers(0, 65535, size=(E, H, 2 * I)).astype(np.uint16)
    t = torch.from_numpy(src.view(np.int16)).cuda().view(torch.bfloat16)
    got = B.pack_w1(t).view(torch.int16).cpu().numpy().view(np.uint16)
    want = np.empty_like(src)
    for p in range(2 * I):
        b, j = divmod(p, 32)
        want[:, :, p] = src[:, :, 16 * b + j] if j < 16 else src[:, :, I + 16 * b + j - 16]
    assert np.array_equal(got, want)


@pytest.mark.parametrize("name", ["tiny", "granite", "qwen", "dsv2lite"])
def test_gemm1_swiglu_parity(gpu_lib, name):
    import torch
    from paper_2609_07536_amd import binding as B
    w = config(name)
    hidden, w1 = layer_inputs(w)
    print(f"{name}: T={w.T} H={w.H} I={w.I} E={w.E} k={w.topk}", flush=True)
    h, _, w1p, _, off, tid, _ = _dev(w, hidden, w1)
    ws = B.Workspace(512)
    x = B.gemm1_swiglu(h, w1p, off, tid, topk=w.topk, rows=w.Mtot, counts=w.counts, workspace=ws)
    torch.cuda.synchronize()
    assert ws.status() == 0
    got = x.view(torch.int16).cpu().numpy().view(np.uint16)
    act, ref_bits = ol.swiglu_reference(hidden, w1, w.expert_offsets, w.token_ids)
    _x_check(got, act, ref_bits, f"{name} x_perm")
    rows = np.random.default_rng(0).choice(w.Mtot, size=min(w.Mtot, 32), replace=False)
    bf = ol.swiglu_rows(hidden, w1, w.expert_offsets, w.token_ids, rows)
    g32 = oc.bf16_bits_to_f32(got[rows]).astype(np.float64)
    assert np.max(np.abs(g32 - bf)) <= 2 ** -7 * np.max(np.abs(bf)) + 1e-6


@pytest.mark.parametrize("name", ["tiny", "granite", "qwen", "dsv2lite"])
def test_layer_forward_parity(gpu_lib, name):
    import torch
    from paper_2609_07536_amd import binding as B
    w = config(name)
    hidden, w1 = layer_inputs(w)
    h, _, w1p, w2, off, tid, g = _dev(w, hidden, w1)
    ref = ol.layer_reference(hidden, w1, w.w2, w.expert_offsets, w.token_ids, w.gate_w, w.T)
    for C in (-1, 0, 5):
        out, used = B.layer_forward(h, w1p, w2, off, tid, g, topk=w.topk, splits=w.L,
                                    counts=w.counts, num_consumers=C)
        torch.cuda.synchronize()
        _check_bar(out.cpu().numpy(), ref, f"{name} layer C={used}")
    # the layer equals its two stages run one after the other, bitwise
    x = B.gemm1_swiglu(h, w1p, off, tid, topk=w.topk, rows=w.Mtot, counts=w.counts)
    out2, _ = B.combine(x, w2, off, tid, g, T=w.T, splits=w.L, topk=w.topk, counts=w.counts,
                        num_consumers=0)
    out1, _ = B.layer_forward(h, w1p, w2, off, tid, g, topk=w.topk, splits=w.L,
                              counts=w.counts, num_consumers=0)
    torch.cuda.synchronize()
    assert np.array_equal(out1.cpu().numpy().view(np.uint32), out2.cpu().numpy().view(np.uint32))


EDGE = [
    # name, T, H, I, E, topk, routing
    ("ragged", 37, 64, 16, 3, 2, ("uniform",)),
    ("I48_partial_tile", 300, 256, 48, 5, 2, ("zipf", 1.0)),
    ("one_expert", 300, 128, 32, 1, 1, ("uniform",)),
    ("H_not_64", 129, 200, 64, 4, 3, ("uniform",)),
    ("H24_single_stage", 50, 24, 16, 2, 1, ("uniform",)),
    ("many_experts", 400, 256, 32, 100, 4, ("zipf", 0.5)),
    ("wide_I", 200, 128, 528, 4, 2, ("uniform",)),
]


@pytest.mark.parametrize("case", EDGE, ids=[c[0] for c in EDGE])
def test_layer_edge_shapes(gpu_lib, case):
    import torch
    from paper_2609_07536_amd import binding as B
    name, T, H, I, E, k, routing = case
    w = custom(T=T, H=H, I=I, E=E, topk=k, L=1, routing=routing, seed=13)
    hidden, w1 = layer_inputs(w)
    h, _, w1p, w2, off, tid, g = _dev(w, hidden, w1)
    x = B.gemm1_swiglu(h, w1p, off, tid, topk=w.topk, rows=w.Mtot, counts=w.counts)
    torch.cuda.synchronize()
    act, ref_bits = ol.swiglu_reference(hidden, w1, w.expert_offsets, w.token_ids)
    _x_check(x.view(torch.int16).cpu().numpy().view(np.uint16), act, ref_bits, f"{name} x_perm")
    ref = ol.layer_reference(hidden, w1, w.w2, w.expert_offsets, w.token_ids, w.gate_w, w.T)
    for C in (-1, 0, 3):
        out, used = B.layer_forward(h, w1p, w2, off, tid, g, topk=w.topk, splits=1,
                                    counts=w.counts, num_consumers=C)
        torch.cuda.synchronize()
        _check_bar(out.cpu().numpy(), ref, f"{name} layer C={used}")


def _random_layer_cases(n=8, seed=7):
    """Seeded random shapes for the up-projection: H a multiple of 8, I of
    16, ragged rows, reductions that are not a multiple of 64 and packed
    widths 2I that are not a multiple of 256."""
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        H = 8 * int(rng.integers(1, 65))
        I = 16 * int(rng.integers(1, 21))
        E = int(rng.integers(1, 25))
        k = int(rng.integers(1, min(E, 6) + 1))
        T = int(rng.integers(1, 400))
        routing = ("uniform",) if i % 2 == 0 else ("zipf", 1.0)
        out.append((f"r{i}_T{T}_H{H}_I{I}_E{E}_k{k}", T, H, I, E, k, routing))
    return out


RANDOM = _random_layer_cases()


@pytest.mark.parametrize("case", RANDOM, ids=[c[0] for c in RANDOM])
def test_layer_random_shapes(gpu_lib, case):
    test_layer_edge_shapes(gpu_lib, case)


def test_layer_dropped_slots_and_bad_token_ids(gpu_lib):
    import torch
    from paper_2609_07536_amd import binding as B
    rng = np.random.default_rng(5)
    T, H, I, E, k = 200, 128, 32, 6, 3
    sel, gates = [], []
    for t in range(T):
        n = int(rng.integers(0, k + 1))
        es = rng.choice([0, 2, 3, 5], size=min(n, 4), replace=False)
        sel.append(list(es))
        gates.append(list(rng.random(len(es)).astype(np.float32)))
    w = explicit(T, H, I, E, sel, gates)
    w.topk = k
    hidden, w1 = layer_inputs(w)
    h, _, w1p, w2, off, tid, g = _dev(w, hidden, w1)
    ref = ol.layer_reference(hidden, w1, w.w2, w.expert_offsets, w.token_ids, w.gate_w, w.T)
    out, _ = B.layer_forward(h, w1p, w2, off, tid, g, topk=k, splits=1, counts=w.counts,
                             num_consumers=0)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    _check_bar(got, ref, "dropped slots")
    empty = [t for t in range(T) if not sel[t]]
    assert np.all(got[empty] == 0)
    # an out-of-range token id: flagged, no fault, the other rows still right
    bad = w.token_ids.copy()
    bad[3] = T + 7
    tid_bad = torch.from_numpy(bad.astype(np.int32)).cuda()
    ws = B.Workspace(512)
    x = B.gemm1_swiglu(h, w1p, off, tid_bad, topk=k, rows=w.Mtot, counts=w.counts, workspace=ws)
    torch.cuda.synchronize()
    assert ws.status(clear=True) == B.MOE_ERR_BAD_ROUTING
    act, ref_bits = ol.swiglu_reference(hidden, w1, w.expert_offsets, w.token_ids)
    keep = np.ones(w.Mtot, dtype=bool)
    keep[3] = False
    _x_check(x.view(torch.int16).cpu().numpy().view(np.uint16)[keep], act[keep], ref_bits[keep],
             "bad id: other rows")
