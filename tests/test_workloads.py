"""The seeded input generator: shapes, routing invariants, determinism."""
import numpy as np
import pytest
import torch

from workloads import (CONFIGS, config, custom, f32_to_bf16_bits,
                       sweep_workloads, zipf_targets)


def _check_layout(w):
    offs = w.expert_offsets.astype(np.int64)
    assert offs[0] == 0 and np.all(np.diff(offs) >= 0)
    assert offs[-1] == w.Mtot == w.token_ids.shape[0] == w.gate_w.shape[0]
    assert np.array_equal(np.diff(offs), w.counts)
    for e in range(w.E):
        seg = w.token_ids[offs[e]:offs[e + 1]]
        assert np.all(np.diff(seg) > 0)          # ascending, distinct tokens
    per_tok = np.bincount(w.token_ids, minlength=w.T)
    assert np.all(per_tok == w.topk)


@pytest.mark.parametrize("name", list(CONFIGS))
def test_configs_layout(name):
    w = config(name, with_tensors=False)
    _check_layout(w)
    assert w.counts.max() <= w.T


def test_config_target_counts():
    g = config("granite", with_tensors=False)
    assert sorted(g.counts.tolist(), reverse=True) == \
        [4096] * 3 + [3309, 2647, 2206, 1891, 1654, 1471, 1324, 1203, 1103,
                      1018, 945, 882, 827]
    assert abs(g.r_expert - 2.0) < 1e-12
    d = config("dsv2lite", with_tensors=False)
    top = sorted(d.counts.tolist(), reverse=True)
    assert top[0] == 4 * (d.T * d.topk // d.E) == 12288
    assert abs(d.r_expert - 4.0) < 1e-12


def test_zipf_targets_properties():
    for total, n, s, cap in [(32768, 16, 1.0, 4096), (32768, 30, 0.8, 8192),
                             (98304, 32, 1.2, 16384), (100, 7, 2.0, 40)]:
        c = zipf_targets(total, n, s, cap)
        assert c.sum() == total and c.max() <= cap
        assert np.all(np.diff(c) <= 1)            # non-increasing up to rounding
        free = (c < cap) & (c >= 100)      # rounding is negligible there
        if free.sum() >= 2:
            idx = np.nonzero(free)[0]
            r0, r1 = idx[0], idx[-1]
            ratio = c[r0] / c[r1]
            want = ((r1 + 1) / (r0 + 1)) ** s
            assert abs(ratio / want - 1) < 0.05


def test_sweep_workloads_layout():
    names = [n for n, _ in sweep_workloads()]
    assert len(names) == 12
    for T in (4096, 32768):
        w = custom(T=T, H=16, I=8, E=32, topk=6, L=2, routing=("zipf", 1.2))
        _check_layout(w)


def test_determinism_per_seed():
    a = custom(T=32, H=16, I=8, E=4, topk=2, seed=5)
    b = custom(T=32, H=16, I=8, E=4, topk=2, seed=5)
    c = custom(T=32, H=16, I=8, E=4, topk=2, seed=6)
    for f in ("x_perm", "w2", "token_ids", "gate_w", "expert_offsets"):
        assert np.array_equal(getattr(a, f), getattr(b, f))
    assert not np.array_equal(a.x_perm, c.x_perm)


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    a = np.concatenate([rng.standard_normal(100000).astype(np.float32),
                        np.float32([0.0, -0.0, 1.0, 1.00390625, 1.01171875,
                                    3.0e-39, -2.5e38])])
    got = f32_to_bf16_bits(a)
    want = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy()
    assert np.array_equal(got.view(np.int16), want)


def test_weight_and_activation_scale():
    w = config("tiny")
    x = (w.x_perm.astype(np.uint32) << 16).view(np.float32)
    W = (w.w2.astype(np.uint32) << 16).view(np.float32)
    assert abs(x.std() - 1.0) < 0.02
    assert abs(W.std() * np.sqrt(w.I) - 1.0) < 0.02
