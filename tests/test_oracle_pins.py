"""Pins for the combine oracle: it is checked against things other than itself.

* the dense, unrouted formula in fp64 (every token against every expert,
  unselected experts weighted by zero);
* the gate invariant (weights of a token sum to one) and its consequence:
  identical experts and identical rows reduce the stage to one plain matrix
  product;
* token relabelling and expert relabelling leave the result unchanged;
* top-1 with unit gates is a plain per-row matrix product; scaling every
  gate scales the output;
* planted mistakes in a copy of the oracle (a shifted expert index, ignored
  gates, a transposed weight) are caught by the dense pin.
"""
import numpy as np
import pytest

from oracle import combine as oc
from workloads import custom, explicit, f32_to_bf16_bits


def _dense_fp64(w):
    """Dense unrouted formula: out = sum_e G[t,e] * (X[t,e,:] @ W2[e])."""
    T, E, I, H = w.T, w.E, w.I, w.H
    x = oc.bf16_bits_to_f32(w.x_perm).astype(np.float64)
    W = oc.bf16_bits_to_f32(w.w2).astype(np.float64)
    rng = np.random.default_rng(1234)
    Xd = rng.standard_normal((T, E, I))      # filler for unselected pairs
    Gd = np.zeros((T, E))
    re = np.repeat(np.arange(E), np.diff(w.expert_offsets))
    for r in range(w.Mtot):
        t, e = int(w.token_ids[r]), int(re[r])
        Xd[t, e] = x[r]
        Gd[t, e] = float(w.gate_w[r])
    return np.einsum("te,teh->th", Gd, np.einsum("tei,eih->teh", Xd, W))


def _ref(w, fn=oc.combine_reference):
    return fn(w.x_perm, w.w2, w.expert_offsets, w.token_ids, w.gate_w, w.T)


@pytest.mark.parametrize("shape", [
    dict(T=12, H=40, I=24, E=4, topk=2),
    dict(T=16, H=64, I=32, E=3, topk=3),
    dict(T=9, H=16, I=48, E=5, topk=1),
])
@pytest.mark.parametrize("routing", [("uniform",), ("zipf", 1.0)])
def test_dense_unrouted_formula(shape, routing):
    w = custom(routing=routing, seed=3, **shape)
    dense = _dense_fp64(w)
    for fn in (oc.combine_reference, oc.combine_bruteforce):
        got = _ref(w, fn)
        assert oc.rel_l2(got, dense) <= 1e-5
        assert np.abs(got - dense).max() <= 1e-5 * np.abs(dense).max()


def test_bruteforce_matches_batched_on_tiny_config():
    from workloads import config
    w = config("tiny")
    a = _ref(w)
    b = _ref(w, oc.combine_bruteforce)
    assert oc.rel_l2(a, b) <= 1e-6


def test_gate_weights_sum_to_one():
    for routing in [("uniform",), ("zipf", 0.8), ("hot_zipf", 4.0, 1.2)]:
        w = custom(T=64, H=8, I=8, E=8, topk=4, routing=routing)
        s = np.zeros(w.T, dtype=np.float64)
        np.add.at(s, w.token_ids, w.gate_w.astype(np.float64))
        assert np.abs(s - 1.0).max() <= w.topk * 2.0 ** -23


def test_identical_experts_reduce_to_one_matmul():
    """All W2_e equal and all k rows of a token equal x_t => out = x @ W."""
    T, H, I, E, k = 20, 24, 16, 4, 3
    w = custom(T=T, H=H, I=I, E=E, topk=k, seed=5)
    rng = np.random.default_rng(9)
    xt = f32_to_bf16_bits(rng.standard_normal((T, I)).astype(np.float32))
    W = f32_to_bf16_bits(rng.standard_normal((I, H)).astype(np.float32))
    w.x_perm = xt[w.token_ids]
    w.w2 = np.broadcast_to(W, (E, I, H)).copy()
    got = _ref(w)
    want = oc.bf16_bits_to_f32(xt).astype(np.float64) @ \
        oc.bf16_bits_to_f32(W).astype(np.float64)
    assert oc.rel_l2(got, want) <= 1e-6


def test_top1_unit_gates_is_per_row_matmul():
    T, H, I, E = 10, 12, 8, 3
    rng = np.random.default_rng(2)
    sel = [[int(rng.integers(E))] for _ in range(T)]
    gates = [[1.0] for _ in range(T)]
    w = explicit(T, H, I, E, sel, gates)
    got = _ref(w)
    x = oc.bf16_bits_to_f32(w.x_perm).astype(np.float64)
    W = oc.bf16_bits_to_f32(w.w2).astype(np.float64)
    re = np.repeat(np.arange(E), np.diff(w.expert_offsets))
    want = np.zeros((T, H))
    for r in range(w.Mtot):
        want[w.token_ids[r]] = x[r] @ W[re[r]]
    assert oc.rel_l2(got, want) <= 1e-6


def test_gate_scaling_is_linear_and_exact_for_powers_of_two():
    w = custom(T=16, H=32, I=16, E=4, topk=2)
    a = _ref(w)
    w.gate_w = (w.gate_w * np.float32(4.0)).astype(np.float32)
    b = _ref(w)
    assert np.array_equal(b, a * np.float32(4.0))


def test_token_relabel_invariance_bitwise():
    w = custom(T=24, H=16, I=8, E=4, topk=2, seed=7)
    a = _ref(w)
    pi = np.random.default_rng(11).permutation(w.T)      # old -> new id
    new_tok = pi[w.token_ids]
    re = np.repeat(np.arange(w.E), np.diff(w.expert_offsets))
    order = np.lexsort((new_tok, re))      # re-sort rows inside each expert
    w.token_ids = new_tok[order].astype(np.int32)
    w.x_perm = w.x_perm[order]
    w.gate_w = w.gate_w[order]
    b = _ref(w)
    assert np.array_equal(b[pi], a)


def test_expert_relabel_invariance():
    w = custom(T=24, H=16, I=8, E=5, topk=2, seed=8)
    a = _ref(w)
    sigma = np.random.default_rng(4).permutation(w.E)   # new expert j = old sigma[j]
    offs = w.expert_offsets.astype(np.int64)
    rows = np.concatenate([np.arange(offs[e], offs[e + 1]) for e in sigma])
    counts = np.diff(offs)[sigma]
    w.expert_offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    w.x_perm = w.x_perm[rows]
    w.token_ids = w.token_ids[rows]
    w.gate_w = w.gate_w[rows]
    w.w2 = w.w2[sigma]
    b = _ref(w)
    assert oc.rel_l2(b, a) <= 1e-6


def test_dropped_slots_and_empty_experts():
    """Tokens with fewer than k (or zero) rows and experts with no rows."""
    T, H, I, E = 6, 8, 8, 4
    sel = [[0, 2], [2], [], [0, 2], [2, 0], [0]]
    gates = [[0.25, 0.75], [1.0], [], [0.5, 0.5], [0.125, 0.875], [1.0]]
    w = explicit(T, H, I, E, sel, gates)
    assert list(w.counts) == [4, 0, 4, 0]
    got = _ref(w)
    assert np.all(got[2] == 0)
    assert oc.rel_l2(got, _dense_fp64(w)) <= 1e-6
    assert oc.rel_l2(_ref(w, oc.combine_bruteforce), got) <= 1e-6


# ---- planted mistakes: a wrong oracle must fail the dense pin -------------

def _wrong_expert_shift(x, w2, offs, tid, g, T):
    return oc.combine_reference(x, np.roll(w2, 1, axis=0), offs, tid, g, T)


def _wrong_ignore_gates(x, w2, offs, tid, g, T):
    return oc.combine_reference(x, w2, offs, tid, np.ones_like(g), T)


def _wrong_transposed_weight(x, w2, offs, tid, g, T):
    return oc.combine_reference(x, np.ascontiguousarray(w2.transpose(0, 2, 1)),
                                offs, tid, g, T)


def _wrong_row_offset(x, w2, offs, tid, g, T):
    return oc.combine_reference(np.roll(x, 1, axis=0), w2, offs, tid, g, T)


@pytest.mark.parametrize("mutant", [_wrong_expert_shift, _wrong_ignore_gates,
                                    _wrong_transposed_weight, _wrong_row_offset])
def test_dense_pin_catches_planted_mistakes(mutant):
    w = custom(T=12, H=16, I=16, E=4, topk=2, seed=3)
    dense = _dense_fp64(w)
    got = mutant(w.x_perm, w.w2, w.expert_offsets, w.token_ids, w.gate_w, w.T)
    assert oc.rel_l2(got, dense) > 1e-2
