"""Pins of the up-projection oracle (grouped GEMM1 + SwiGLU) and of the
whole post-router layer, against what the mathematics fixes: a dense fp64
formula, closed forms of silu, zero projections, the token gather, an
independent bf16 rounding check, and planted mistakes that must fail."""
import numpy as np
import pytest
from scipy.special import expit

from oracle import combine as oc
from oracle import layer as ol
from workloads import custom, explicit, f32_to_bf16_bits, layer_inputs


def _tiny(seed=5, T=7, H=24, I=16, E=3, k=2):
    w = custom(T=T, H=H, I=I, E=E, topk=k, L=1, routing=("uniform",), seed=seed)
    hidden, w1 = layer_inputs(w)
    return w, hidden, w1


def _dense_act(hidden_bits, w1_bits, offsets, token_ids):
    """fp64, no per-expert grouping: every row against every expert, then the
    one-hot expert mask selects."""
    h = oc.bf16_bits_to_f32(hidden_bits).astype(np.float64)
    w1 = oc.bf16_bits_to_f32(w1_bits).astype(np.float64)
    E, _, two_i = w1.shape
    I = two_i // 2
    rows = int(offsets[-1])
    mask = np.zeros((rows, E))
    for e in range(E):
        mask[offsets[e]:offsets[e + 1], e] = 1.0
    hr = h[np.asarray(token_ids, dtype=np.int64)]
    g_all = np.einsum("rh,ehi->rei", hr, w1[:, :, :I])
    u_all = np.einsum("rh,ehi->rei", hr, w1[:, :, I:])
    g = np.einsum("re,rei->ri", mask, g_all)
    u = np.einsum("re,rei->ri", mask, u_all)
    return g * expit(g) * u


def test_silu_closed_forms():
    z = np.linspace(-30, 30, 601)
    np.testing.assert_allclose(ol.silu(z), z * expit(z), rtol=1e-13, atol=1e-300)
    assert ol.silu(np.float64(0.0)) == 0.0
    assert ol.silu(np.float64(40.0)) == 40.0
    assert -1e-15 < ol.silu(np.float64(-40.0)) < 0.0
    assert ol.silu(np.float32(-200.0)) == 0.0          # exp overflow: the limit
    # silu(z) - silu(-z) = z
    np.testing.assert_allclose(ol.silu(z) - ol.silu(-z), z, atol=1e-12)


def test_swiglu_matches_dense_fp64_formula():
    w, hidden, w1 = _tiny()
    act, bits = ol.swiglu_reference(hidden, w1, w.expert_offsets, w.token_ids)
    dense = _dense_act(hidden, w1, w.expert_offsets, w.token_ids)
    np.testing.assert_allclose(act, dense, rtol=2e-5, atol=2e-6)
    rows = np.arange(w.Mtot)
    np.testing.assert_allclose(ol.swiglu_rows(hidden, w1, w.expert_offsets, w.token_ids, rows),
                               dense, rtol=1e-12, atol=1e-12)


def test_zero_gate_or_up_projection_gives_zero():
    w, hidden, w1 = _tiny(seed=6)
    I = w.I
    wg0 = w1.copy()
    wg0[:, :, :I] = 0
    act, bits = ol.swiglu_reference(hidden, wg0, w.expert_offsets, w.token_ids)
    assert np.all(act == 0) and np.all((bits & 0x7FFF) == 0)
    wu0 = w1.copy()
    wu0[:, :, I:] = 0
    act, _ = ol.swiglu_reference(hidden, wu0, w.expert_offsets, w.token_ids)
    assert np.all(act == 0)


def test_gather_follows_token_ids():
    """Relabelling the tokens (and permuting the hidden rows with them)
    leaves every routed row's activation bitwise unchanged."""
    w, hidden, w1 = _tiny(seed=7, T=9)
    perm = np.random.default_rng(1).permutation(w.T)
    hidden2 = np.empty_like(hidden)
    hidden2[perm] = hidden
    tid2 = perm[w.token_ids].astype(np.int32)
    a1, b1 = ol.swiglu_reference(hidden, w1, w.expert_offsets, w.token_ids)
    a2, b2 = ol.swiglu_reference(hidden2, w1, w.expert_offsets, tid2)
    assert np.array_equal(b1, b2) and np.array_equal(a1.view(np.uint32), a2.view(np.uint32))


def _nearest_bf16(x: float) -> int:
    """Independent rounding: the two bf16 neighbours of x by truncation, the
    nearer one, ties to the even pattern."""
    u = int(np.float32(x).view(np.uint32))
    lo = u >> 16
    cands = [lo, lo + 1]
    # an infinite neighbour stands for +-2^128 (the IEEE overflow threshold is
    # the midpoint between the largest finite value and 2^128)
    vals = [float(np.uint32(c << 16).view(np.float32)) for c in cands]
    vals = [np.copysign(2.0 ** 128, v) if np.isinf(v) else v for v in vals]
    d = [abs(v - float(np.float32(x))) for v in vals]
    if d[0] < d[1]:
        return cands[0]
    if d[1] < d[0]:
        return cands[1]
    return cands[0] if cands[0] % 2 == 0 else cands[1]


def test_rounding_is_nearest_even():
    rng = np.random.default_rng(3)
    x = np.concatenate([rng.standard_normal(2000).astype(np.float32) * 10,
                        # exact ties: a bf16 value plus half an ulp
                        (np.arange(1, 200, dtype=np.uint32) << np.uint32(16) | np.uint32(0x8000))
                        .astype(np.uint32).view(np.float32) * np.float32(1.0),
                        np.float32([0.0, -0.0, 1e-40, -3.4e38])])
    x = x[np.isfinite(x)]
    got = ol.round_to_bf16_bits(x)
    want = np.array([_nearest_bf16(v) for v in x], dtype=np.int64)
    assert np.array_equal(got.astype(np.int64), want)


def test_planted_mistakes_fail_the_dense_pin():
    w, hidden, w1 = _tiny(seed=8)
    dense = _dense_act(hidden, w1, w.expert_offsets, w.token_ids)
    I = w.I
    # gate and up swapped
    sw = np.concatenate([w1[:, :, I:], w1[:, :, :I]], axis=2)
    a, _ = ol.swiglu_reference(hidden, sw, w.expert_offsets, w.token_ids)
    assert not np.allclose(a, dense, rtol=1e-3, atol=1e-3)
    # no gather: row r reads hidden row r % T
    tid_bad = (np.arange(w.Mtot) % w.T).astype(np.int32)
    a, _ = ol.swiglu_reference(hidden, w1, w.expert_offsets, tid_bad)
    assert not np.allclose(a, dense, rtol=1e-3, atol=1e-3)
    # expert shifted by one
    off = w.expert_offsets
    a, _ = ol.swiglu_reference(hidden, np.roll(w1, 1, axis=0), off, w.token_ids)
    assert not np.allclose(a, dense, rtol=1e-3, atol=1e-3)


def test_layer_matches_dense_formula_within_bf16_staging():
    """End to end on a tiny input: the layer oracle against the fp64 formula
    sum_j g_j * (silu(h Wg) * (h Wu)) @ W2, whose only difference is the bf16
    rounding of the activation."""
    w, hidden, w1 = _tiny(seed=9, T=11, H=32, I=16, E=4, k=2)
    out = ol.layer_reference(hidden, w1, w.w2, w.expert_offsets, w.token_ids, w.gate_w, w.T)
    act = _dense_act(hidden, w1, w.expert_offsets, w.token_ids)
    w2 = oc.bf16_bits_to_f32(w.w2).astype(np.float64)
    e_of = oc.row_experts(w.expert_offsets)
    ref = np.zeros((w.T, w.H))
    for r in range(w.Mtot):
        ref[w.token_ids[r]] += w.gate_w[r] * (act[r] @ w2[e_of[r]])
    assert oc.rel_l2(out, ref) <= 5e-3
    assert np.max(np.abs(out - ref)) <= 1e-2 * np.max(np.abs(ref))


def test_layer_with_dropped_slots():
    """Tokens without rows get zeros; experts without rows are skipped."""
    sel = [[0, 2], [], [2], [0], []]
    gates = [[0.6, 0.4], [], [1.0], [1.0], []]
    w = explicit(5, 16, 16, 3, sel, gates)
    hidden, w1 = layer_inputs(w)
    out = ol.layer_reference(hidden, w1, w.w2, w.expert_offsets, w.token_ids, w.gate_w, w.T)
    assert np.all(out[[1, 4]] == 0)
    assert np.any(out[[0, 2, 3]] != 0)


def test_generator_layer_inputs_are_bf16_of_the_recipe():
    w = custom(T=4, H=8, I=16, E=2, topk=1, L=1, seed=2)
    hidden, w1 = layer_inputs(w)
    assert hidden.shape == (4, 8) and w1.shape == (2, 8, 32)
    assert hidden.dtype == np.uint16 and w1.dtype == np.uint16
    # the weights' scale: N(0, 1/H), so |w| is far below 1 for H = 8
    assert np.abs(oc.bf16_bits_to_f32(w1)).max() < 3.0
    h2, w12 = layer_inputs(w)
    assert np.array_equal(hidden, h2) and np.array_equal(w1, w12)
