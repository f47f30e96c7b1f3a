"""CPU oracle for the MoE GEMM2 + gate-weighted combine (test infrastructure).

Only tests, the smoke check and the benchmark's CPU-baseline leg use this
module; the product path never imports it.

What is computed (Background, "Distributed MoE Execution", third step: the
grouped GEMM2 projects each expert's intermediate rows back to the hidden
size, and the combine aggregates each token's top-k expert contributions):

    Y[r, :]  = x_perm[r, :] @ W2[e(r)]           e(r): offsets[e] <= r < offsets[e+1]
    out[t, :] = sum over rows r with token_ids[r] == t of gate_w[r] * Y[r, :]

The partition of the GPU between compute and consumer workgroups (the paper's
decision variable C) never changes this result (Method, "System Integration
and Correctness": only C and the resulting reservation differ), so the
oracle is the plain definition written out.  Arithmetic is fp32 with bf16
inputs widened exactly; the k contributions of a token are summed in
ascending permuted-row order.  Pins (tests/test_oracle_pins.py) tie it to a
dense fp64 formula, to gate and permutation invariants and to a plain
matrix product in the special cases that reduce to one; the bf16 widening
and the two acceptance measures (rel_l2, max_abs_ratio) are pinned on their
own (tests/test_oracle_numeric_pins.py: every bf16 pattern against torch's
conversion, hand-decoded values, hand-worked arrays, planted mistakes).
"""
from __future__ import annotations

import numpy as np


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to fp32 (exact: bf16 is the top half of fp32)."""
    b = np.ascontiguousarray(bits).view(np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def row_experts(offsets: np.ndarray) -> np.ndarray:
    """e(r) for every permuted row r, from the expert offsets."""
    offsets = np.asarray(offsets, dtype=np.int64)
    counts = np.diff(offsets)
    if (counts < 0).any():
        raise ValueError("expert offsets must be non-decreasing")
    return np.repeat(np.arange(counts.shape[0]), counts)


def _rows_by_token(token_ids: np.ndarray, T: int):
    """For each token, its rows in ascending order, as (order, start, count)."""
    tid = np.asarray(token_ids, dtype=np.int64)
    if tid.size and (tid.min() < 0 or tid.max() >= T):
        raise ValueError("token id out of range")
    order = np.lexsort((np.arange(tid.size), tid))   # by token, then row
    count = np.bincount(tid, minlength=T)
    start = np.zeros(T + 1, dtype=np.int64)
    start[1:] = np.cumsum(count)
    return order, start, count


def combine_reference(x_bits, w2_bits, offsets, token_ids, gate_w, T,
                      dtype=np.float32) -> np.ndarray:
    """out[T, H]: per-expert products, then the per-token weighted sum.

    Each expert's rows are multiplied by that expert's weights in one matrix
    product (a library primitive); the token sum then adds the j-th row of
    every token in ascending row order, j = 0, 1, ...
    """
    x = bf16_bits_to_f32(x_bits).astype(dtype, copy=False)
    w2 = bf16_bits_to_f32(w2_bits).astype(dtype, copy=False)
    offsets = np.asarray(offsets, dtype=np.int64)
    E, H = w2.shape[0], w2.shape[2]
    Mtot = int(offsets[-1])
    Y = np.empty((Mtot, H), dtype=dtype)
    for e in range(E):
        a, b = int(offsets[e]), int(offsets[e + 1])
        if b > a:
            Y[a:b] = x[a:b] @ w2[e]
    g = np.asarray(gate_w, dtype=dtype)
    order, start, count = _rows_by_token(token_ids, T)
    out = np.zeros((T, H), dtype=dtype)
    kmax = int(count.max()) if T else 0
    toks = np.arange(T)
    for j in range(kmax):
        have = count > j
        t = toks[have]
        r = order[start[:-1][have] + j]
        out[t] += g[r][:, None] * Y[r]
    return out


def combine_tokens(x_bits, w2_bits, offsets, token_ids, gate_w, T, tokens,
                   dtype=np.float32) -> np.ndarray:
    """Brute force for selected tokens: sum_j g_j * (x_j @ W2[e_j]).

    Walks token by token and row by row (ascending), one vector-matrix
    product per routed row; used on small inputs and on sampled tokens of
    large ones.
    """
    offsets = np.asarray(offsets, dtype=np.int64)
    H = w2_bits.shape[2]
    re = row_experts(offsets)
    order, start, count = _rows_by_token(token_ids, T)
    g = np.asarray(gate_w, dtype=dtype)
    out = np.zeros((len(tokens), H), dtype=dtype)
    for i, t in enumerate(tokens):
        acc = np.zeros(H, dtype=dtype)
        for j in range(int(count[t])):
            r = int(order[start[t] + j])
            xr = bf16_bits_to_f32(x_bits[r]).astype(dtype)
            we = bf16_bits_to_f32(w2_bits[re[r]]).astype(dtype)
            acc = acc + g[r] * (xr @ we)
        out[i] = acc
    return out


def combine_bruteforce(x_bits, w2_bits, offsets, token_ids, gate_w, T,
                       dtype=np.float32) -> np.ndarray:
    return combine_tokens(x_bits, w2_bits, offsets, token_ids, gate_w, T,
                          range(T), dtype=dtype)


def rel_l2(got: np.ndarray, ref: np.ndarray) -> float:
    ref64 = ref.astype(np.float64)
    den = np.linalg.norm(ref64)
    num = np.linalg.norm(got.astype(np.float64) - ref64)
    return float(num / den) if den > 0 else float(num)


def max_abs_ratio(got: np.ndarray, ref: np.ndarray) -> float:
    """max|got - ref| / max|ref| (the elementwise acceptance measure)."""
    m = float(np.abs(ref).max()) if ref.size else 0.0
    d = float(np.abs(got.astype(np.float64) - ref).max()) if ref.size else 0.0
    return d / m if m > 0 else d


# Acceptance bar for bf16 inputs with fp32 accumulation.
REL_L2_TOL = 5e-3
MAX_ABS_TOL = 1e-2
