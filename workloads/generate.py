"""Seeded synthetic inputs for the MoE down-projection + combine stage.

This module only draws and lays out inputs; it holds none of the stage's
arithmetic (no GEMM, no reduction, no selector).  Both the CPU oracle and the
GPU path consume what it returns, so every array here is plain numpy.

Shapes follow the models the paper evaluates (Table "MoE model
configurations", experimental setup): hidden size H, expert FFN size F split
by tensor parallelism into the local reduction size I, routed experts E split
by expert parallelism into local experts, and top-k.  The paper measures on
router traces that are not available here; the routings below stand in for
them (uniform top-k of iid logits, and Zipf-skewed expert loads), and each
workload records the skew statistic R_expert = max_e L_e / (M k / E) that the
paper uses to pick its p50/p90 traces.

Draw recipe (fixed, so every consumer sees the same bits for a seed):
  * independent streams ``default_rng([seed, cfg_id, stream])`` for the
    activations, the weights, the router logits and the routing decisions;
  * activations x_perm ~ N(0, 1) and weights W2 ~ N(0, 1/I), drawn in fp32
    and rounded to bf16 with round-to-nearest-even, returned as uint16 bit
    patterns;
  * router logits ~ N(0, 1) [T, E]; probabilities by softmax in fp64;
  * uniform routing: each token takes the top-k probabilities (ties to the
    lower expert index);
  * skewed routing: deterministic per-expert target counts (Zipf over a
    seeded expert->rank permutation, capped at T with water-filling and
    rounded by largest remainder), realised by a greedy assignment that gives
    each token (in seeded random order) the k experts with the most remaining
    capacity (ties broken by seeded noise); this greedy never gets stuck
    because no expert ever needs more tokens than remain;
  * gate weights: the chosen experts' softmax probabilities, renormalised to
    sum to one per token, stored as fp32;
  * rows grouped by expert (expert-major), ascending token id inside an
    expert; expert_offsets is the exclusive prefix sum of the counts;
  * for the whole post-router layer (``layer_inputs``): hidden states
    ~ N(0, 1) [T, H] and the up-projection weights ~ N(0, 1/H) [E, H, 2I]
    (columns 0..I-1 the gate projection, I..2I-1 the up projection), each
    from its own stream, rounded to bf16 the same way.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Tuple

import numpy as np

# Stream ids for default_rng([seed, cfg_id, stream]).
_S_X, _S_W2, _S_LOGITS, _S_ROUTE = 1, 2, 3, 4
_S_HIDDEN, _S_W1 = 5, 6


@dataclasses.dataclass
class Workload:
    name: str
    T: int            # tokens (M in the paper's notation, one GPU so D = 1)
    H: int            # hidden size: GEMM2 output dim N
    I: int            # local expert intermediate size: GEMM2 reduction dim K
    E: int            # local experts
    topk: int
    L: int            # pipeline splits along H
    routing: Tuple    # ("uniform",) | ("zipf", s) | ("hot_zipf", factor, s)
    seed: int
    x_perm: np.ndarray         # uint16 bf16 bits [Mtot, I]
    w2: np.ndarray             # uint16 bf16 bits [E, I, H]
    expert_offsets: np.ndarray  # int32 [E+1]
    token_ids: np.ndarray      # int32 [Mtot]
    gate_w: np.ndarray         # float32 [Mtot]
    counts: np.ndarray         # int64 [E]

    @property
    def Mtot(self) -> int:
        return int(self.expert_offsets[-1])

    @property
    def r_expert(self) -> float:
        mean = self.T * self.topk / self.E
        return float(self.counts.max() / mean) if mean > 0 else 0.0

    @property
    def flops(self) -> int:
        """2 * routed rows * I * H: only routed rows, no tile padding."""
        return 2 * self.Mtot * self.I * self.H


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (nearest, ties to even); finite inputs only."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def _rng(seed: int, cfg_id: int, stream: int) -> np.random.Generator:
    return np.random.default_rng([seed, cfg_id, stream])


def zipf_targets(total: int, n: int, s: float, cap: int) -> np.ndarray:
    """Integer loads by rank (rank 0 hottest), proportional to (r+1)^-s.

    Loads above ``cap`` are clipped and the excess is re-spread over the
    unclipped ranks in proportion to their weights (water-filling), then the
    real targets are rounded by largest remainder so they sum to ``total``.
    Requires total <= n * cap.
    """
    if total > n * cap:
        raise ValueError("infeasible: total exceeds n * cap")
    w = np.arange(1, n + 1, dtype=np.float64) ** (-float(s))
    capped = np.zeros(n, dtype=bool)
    while True:
        free = ~capped
        remaining = total - cap * int(capped.sum())
        t = np.zeros(n, dtype=np.float64)
        t[capped] = cap
        t[free] = remaining * w[free] / w[free].sum()
        over = free & (t > cap)
        if not over.any():
            break
        capped |= over
    base = np.floor(t).astype(np.int64)
    base = np.minimum(base, cap)
    short = total - int(base.sum())
    frac = t - base
    # hand out the missing units to the largest fractional parts that are
    # still below the cap (ties to the hotter rank)
    order = sorted(range(n), key=lambda r: (-frac[r], r))
    i = 0
    while short > 0:
        r = order[i % n]
        if base[r] < cap:
            base[r] += 1
            short -= 1
        i += 1
    return base


def target_counts(routing: Tuple, T: int, E: int, topk: int,
                  rng: np.random.Generator) -> np.ndarray:
    """Per-expert target loads for the skewed routings, indexed by expert."""
    total = T * topk
    kind = routing[0]
    perm = rng.permutation(E)          # perm[rank] = expert id
    if kind == "zipf":
        by_rank = zipf_targets(total, E, routing[1], T)
    elif kind == "hot_zipf":
        factor, s = routing[1], routing[2]
        hot = min(T, int(round(factor * total / E)))
        rest = zipf_targets(total - hot, E - 1, s, hot)
        by_rank = np.concatenate([[hot], rest])
    else:
        raise ValueError(f"unknown routing {routing!r}")
    counts = np.zeros(E, dtype=np.int64)
    counts[perm] = by_rank
    return counts


def _assign_by_targets(counts: np.ndarray, T: int, topk: int,
                       rng: np.random.Generator) -> np.ndarray:
    """[T, topk] expert ids realising ``counts`` exactly (distinct per token)."""
    E = counts.shape[0]
    rem = counts.astype(np.float64).copy()
    order = rng.permutation(T)
    noise = rng.random((T, E)) * 0.5     # < 1: only reorders equal loads
    sel = np.empty((T, topk), dtype=np.int64)
    for t in order:
        key = rem + noise[t]
        top = np.argpartition(-key, topk - 1)[:topk]
        if np.any(rem[top] <= 0):
            raise RuntimeError("assignment infeasible")  # cannot happen
        rem[top] -= 1
        sel[t] = np.sort(top)
    assert not rem.any()
    return sel


def make_workload(name: str, T: int, H: int, I: int, E: int, topk: int,
                  L: int, routing: Tuple, seed: int = 0, cfg_id: int = 0,
                  with_tensors: bool = True) -> Workload:
    if not (1 <= topk <= E):
        raise ValueError("need 1 <= topk <= E")
    logits = _rng(seed, cfg_id, _S_LOGITS).standard_normal((T, E))
    z = logits - logits.max(axis=1, keepdims=True)
    p = np.exp(z)
    p /= p.sum(axis=1, keepdims=True)
    if routing[0] == "uniform":
        # stable sort on -p: equal probabilities keep the lower expert first
        sel = np.sort(np.argsort(-p, axis=1, kind="stable")[:, :topk], axis=1)
    else:
        rr = _rng(seed, cfg_id, _S_ROUTE)
        counts_t = target_counts(routing, T, E, topk, rr)
        sel = _assign_by_targets(counts_t, T, topk, rr)
    g = np.take_along_axis(p, sel, axis=1)
    g = (g / g.sum(axis=1, keepdims=True)).astype(np.float32)

    tok = np.repeat(np.arange(T, dtype=np.int64), topk)
    exp = sel.reshape(-1)
    gflat = g.reshape(-1)
    order = np.lexsort((tok, exp))       # expert-major, token ascending
    token_ids = tok[order].astype(np.int32)
    gate_w = gflat[order].astype(np.float32)
    counts = np.bincount(exp, minlength=E).astype(np.int64)
    offsets = np.zeros(E + 1, dtype=np.int32)
    offsets[1:] = np.cumsum(counts)
    Mtot = int(offsets[-1])

    if with_tensors:
        x = _rng(seed, cfg_id, _S_X).standard_normal((Mtot, I), dtype=np.float32)
        x_perm = f32_to_bf16_bits(x)
        del x
        w = _rng(seed, cfg_id, _S_W2).standard_normal((E, I, H), dtype=np.float32)
        w *= np.float32(1.0 / np.sqrt(I))
        w2 = f32_to_bf16_bits(w)
        del w
    else:
        x_perm = np.zeros((0, I), dtype=np.uint16)
        w2 = np.zeros((0, I, H), dtype=np.uint16)
    return Workload(name=name, T=T, H=H, I=I, E=E, topk=topk, L=L,
                    routing=tuple(routing), seed=seed, x_perm=x_perm, w2=w2,
                    expert_offsets=offsets, token_ids=token_ids,
                    gate_w=gate_w, counts=counts)


# The evaluated shapes, one GPU's share of each model (TP-split I, EP-split
# E), with the paper's split counts (one split for the H = 1024 model, two
# for the H = 2048 models).
CONFIGS: Dict[str, dict] = {
    "tiny": dict(T=256, H=1024, I=512, E=8, topk=2, L=1,
                 routing=("uniform",), cfg_id=1),
    "granite": dict(T=4096, H=1024, I=256, E=16, topk=8, L=1,
                    routing=("zipf", 1.0), cfg_id=2),
    "qwen": dict(T=8192, H=2048, I=704, E=30, topk=4, L=2,
                 routing=("zipf", 0.8), cfg_id=3),
    "dsv2lite": dict(T=16384, H=2048, I=704, E=32, topk=6, L=2,
                     routing=("hot_zipf", 4.0, 1.2), cfg_id=4),
}

CONFIG_TITLES = {
    "tiny": "Tiny MoE down-proj+combine (T=256,H=1024,I=512,E=8,top-2)",
    "granite": "Granite-like one-GPU share (T=4096,H=1024,I=256,E=16,top-8,Zipf1.0)",
    "qwen": "Qwen-MoE-like share (T=8192,H=2048,I=704,E=30,top-4,Zipf0.8)",
    "dsv2lite": "DeepSeek-V2-Lite-like share (T=16384,H=2048,I=704,E=32,top-6,hot4x+Zipf1.2)",
}

SWEEP_T = (4096, 8192, 16384, 32768)
SWEEP_SKEW = (("uniform",), ("zipf", 0.8), ("zipf", 1.2))


def config(name: str, seed: int = 0, with_tensors: bool = True) -> Workload:
    c = dict(CONFIGS[name])
    cfg_id = c.pop("cfg_id")
    return make_workload(name, seed=seed, cfg_id=cfg_id,
                         with_tensors=with_tensors, **c)


def sweep_workloads() -> List[Tuple[str, dict]]:
    """The selector sweep: DeepSeek-V2-Lite-like shapes over T and skew."""
    out = []
    for T in SWEEP_T:
        for sk in SWEEP_SKEW:
            tag = "uniform" if sk[0] == "uniform" else f"zipf{sk[1]}"
            out.append((f"sweep_T{T}_{tag}",
                        dict(T=T, H=2048, I=704, E=32, topk=6, L=2,
                             routing=sk, cfg_id=5)))
    return out


def sweep_workload(name: str, seed: int = 0,
                   with_tensors: bool = True) -> Workload:
    for n, c in sweep_workloads():
        if n == name:
            c = dict(c)
            cfg_id = c.pop("cfg_id")
            return make_workload(n, seed=seed, cfg_id=cfg_id,
                                 with_tensors=with_tensors, **c)
    raise KeyError(name)


def custom(T: int, H: int, I: int, E: int, topk: int, L: int = 1,
           routing: Tuple = ("uniform",), seed: int = 0,
           cfg_id: int = 99) -> Workload:
    return make_workload("custom", T=T, H=H, I=I, E=E, topk=topk, L=L,
                         routing=routing, seed=seed, cfg_id=cfg_id)


def explicit(T: int, H: int, I: int, E: int, sel: np.ndarray,
             gates: np.ndarray, L: int = 1, seed: int = 0,
             cfg_id: int = 98, name: str = "explicit") -> Workload:
    """Workload from an explicit routing: sel[t] lists the experts of token
    t (ragged lists allowed, each with distinct experts), gates[t] their
    weights.  Tokens may have fewer entries than others (dropped slots)."""
    tok, exp, gw = [], [], []
    for t in range(T):
        for e, g in zip(sel[t], gates[t]):
            tok.append(t)
            exp.append(int(e))
            gw.append(float(g))
    tok = np.asarray(tok, dtype=np.int64)
    exp = np.asarray(exp, dtype=np.int64)
    gw = np.asarray(gw, dtype=np.float32)
    order = np.lexsort((tok, exp))
    counts = np.bincount(exp, minlength=E).astype(np.int64)
    offsets = np.zeros(E + 1, dtype=np.int32)
    offsets[1:] = np.cumsum(counts)
    Mtot = int(offsets[-1])
    topk = max((len(s) for s in sel), default=1)
    x = _rng(seed, cfg_id, _S_X).standard_normal((Mtot, I), dtype=np.float32)
    w = _rng(seed, cfg_id, _S_W2).standard_normal((E, I, H), dtype=np.float32)
    w *= np.float32(1.0 / np.sqrt(I))
    return Workload(name=name, T=T, H=H, I=I, E=E, topk=max(topk, 1), L=L,
                    routing=("explicit",), seed=seed,
                    x_perm=f32_to_bf16_bits(x), w2=f32_to_bf16_bits(w),
                    expert_offsets=offsets,
                    token_ids=tok[order].astype(np.int32),
                    gate_w=gw[order], counts=counts)


def layer_inputs(w: Workload):
    """Hidden states bf16 [T, H] and up-projection weights bf16 [E, H, 2I]
    (gate columns, then up columns) for workload w, as uint16 bit patterns."""
    h = _rng(w.seed, _cfg_of(w), _S_HIDDEN).standard_normal((w.T, w.H), dtype=np.float32)
    hidden = f32_to_bf16_bits(h)
    del h
    g = _rng(w.seed, _cfg_of(w), _S_W1).standard_normal((w.E, w.H, 2 * w.I), dtype=np.float32)
    g *= np.float32(1.0 / np.sqrt(w.H))
    w1 = f32_to_bf16_bits(g)
    del g
    return hidden, w1


def _cfg_of(w: Workload) -> int:
    """The stream id of a workload's configuration (a hash of its name for
    workloads outside the named configurations)."""
    if w.name in CONFIGS:
        return CONFIGS[w.name]["cfg_id"]
    return 1000 + sum(ord(c) for c in w.name) % 1000
