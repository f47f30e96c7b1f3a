"""CPU oracle for the up-projection (grouped GEMM1 with the SwiGLU
activation) and the whole post-router layer (test infrastructure).

Only tests, the smoke check and the benchmark's CPU-baseline leg use this
module; the product path never imports it and shares no code with it.

What is computed (Background, "Distributed MoE Execution": after the router,
each expert's grouped GEMM1 computes the gate and up projections of its
routed tokens, the gated activation combines them, GEMM2 projects back to
the hidden size and the combine aggregates each token's top-k
contributions):

    h_r          = hidden[token_ids[r], :]
    x_perm[r, c] = silu(h_r @ Wg[e(r)])[c] * (h_r @ Wu[e(r)])[c],   silu(z) = z / (1 + exp(-z))
    out          = the down-projection and combine of x_perm (oracle.combine)

W1[e] is [H, 2I]: columns 0..I-1 are Wg[e], columns I..2I-1 are Wu[e].  The
products are fp32 with bf16 inputs widened exactly, the activation is fp32,
and x_perm is rounded once to bf16 (round to nearest, ties to even), the
precision the down-projection reads.  Pins: tests/test_layer_oracle.py (a
dense fp64 formula, closed forms of silu, zero projections, the gather, an
independent rounding check).
"""
from __future__ import annotations

import numpy as np

from .combine import bf16_bits_to_f32, combine_reference, row_experts


def silu(z: np.ndarray) -> np.ndarray:
    """z / (1 + exp(-z)) in the dtype of z (exp overflow gives -0 for very
    negative z, the limit)."""
    with np.errstate(over="ignore"):
        return z / (1 + np.exp(-z))


def round_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round to nearest, ties to even (NaN stays
    NaN)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)).astype(np.uint16)
    nan = np.isnan(np.asarray(a, dtype=np.float32))
    r[nan] = ((u[nan] >> np.uint64(16)).astype(np.uint16) | np.uint16(0x40))
    return r


def swiglu_reference(hidden_bits, w1_bits, offsets, token_ids):
    """(act fp32 [rows, I], x_perm bf16 bits [rows, I]) for every routed row:
    per expert, the gathered hidden rows times the gate and the up halves of
    its weights (library matrix products), then silu(gate) * up."""
    hidden = bf16_bits_to_f32(hidden_bits)
    w1 = bf16_bits_to_f32(w1_bits)
    offsets = np.asarray(offsets, dtype=np.int64)
    tid = np.asarray(token_ids, dtype=np.int64)
    E, _, two_i = w1.shape
    I = two_i // 2
    rows = int(offsets[-1])
    act = np.zeros((rows, I), dtype=np.float32)
    for e in range(E):
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        if hi <= lo:
            continue
        h = hidden[tid[lo:hi]]
        g = h @ w1[e][:, :I]
        u = h @ w1[e][:, I:]
        act[lo:hi] = silu(g) * u
    return act, round_to_bf16_bits(act)


def swiglu_rows(hidden_bits, w1_bits, offsets, token_ids, rows) -> np.ndarray:
    """Brute force in fp64 for selected rows: one vector-matrix product per
    row with its expert's gate and up weights."""
    hidden = bf16_bits_to_f32(hidden_bits).astype(np.float64)
    w1 = bf16_bits_to_f32(w1_bits)
    e_of = row_experts(offsets)
    I = w1.shape[2] // 2
    out = np.zeros((len(rows), I), dtype=np.float64)
    for i, r in enumerate(rows):
        h = hidden[int(token_ids[r])]
        w = w1[e_of[r]].astype(np.float64)
        g = h @ w[:, :I]
        u = h @ w[:, I:]
        out[i] = g / (1 + np.exp(-g)) * u
    return out


def layer_reference(hidden_bits, w1_bits, w2_bits, offsets, token_ids, gate_w, T) -> np.ndarray:
    """out [T, H] fp32 of the whole post-router layer."""
    _, x_bits = swiglu_reference(hidden_bits, w1_bits, offsets, token_ids)
    return combine_reference(x_bits, w2_bits, offsets, token_ids, gate_w, T)
