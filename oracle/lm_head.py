"""Oracle of the LM head fused with the vocabulary argmax (TEST
INFRASTRUCTURE ONLY): the target model's logits of every tree node are the
node's final hidden state times the LM-head weight (the same one-pass GEMM the
paper applies on the draft side, §4.2: k matrix-vector products as one
matrix product), and verification needs only each row's argmax (greedy
decoding, §7.1), so the logits never have to be stored.

Arithmetic: bf16 inputs; the products are exact and the sums are taken in fp64
(numpy matmul of the fp64 values), which is the exact logit up to fp64
rounding. Argmax: largest value, lowest vocabulary id on ties.

`margin` reports, per row, the gap between the largest and the second largest
logit and `scale` the row's sum of |h_i w_i| over the winning entry, so a
caller can tell whether a reduced-precision evaluation (fp32 sums) is bound to
find the same winner.
"""
from __future__ import annotations

import numpy as np

from .tree_build import bf16_bits_to_f32


def lm_head_logits(hidden_bits: np.ndarray, w_bits: np.ndarray) -> np.ndarray:
    """[R, d] x [V, d] bf16 -> [R, V] fp64 logits (exact products, fp64 sums)."""
    h = bf16_bits_to_f32(hidden_bits).astype(np.float64)
    w = bf16_bits_to_f32(w_bits).astype(np.float64)
    return h @ w.T


def lm_head_argmax(hidden_bits: np.ndarray, w_bits: np.ndarray, chunk: int = 8192):
    """Per-row argmax of hidden @ W^T (lowest id on ties), its top-2 margin and
    the magnitude sum(|h_i w_i|) of the two competing entries (their maximum).

    hidden_bits [R, d] uint16, w_bits [V, d] uint16. The vocabulary is taken in
    chunks so that only [R, chunk] logits exist at a time."""
    hidden_bits = np.asarray(hidden_bits, dtype=np.uint16)
    w_bits = np.asarray(w_bits, dtype=np.uint16)
    R = hidden_bits.shape[0]
    V = w_bits.shape[0]
    h = bf16_bits_to_f32(hidden_bits).astype(np.float64)
    top_v = np.full((R, 2), -np.inf)                 # running two largest (value, id)
    top_i = np.full((R, 2), np.iinfo(np.int64).max, dtype=np.int64)
    rows = np.arange(R)[:, None]
    for v0 in range(0, V, chunk):
        w = bf16_bits_to_f32(w_bits[v0:v0 + chunk]).astype(np.float64)
        lg = h @ w.T                                              # [R, c]
        c2 = np.argsort(-lg, axis=1, kind="stable")[:, :2]        # lowest id first among equals
        cand_v = np.concatenate([top_v, lg[rows, c2]], axis=1)
        cand_i = np.concatenate([top_i, c2 + v0], axis=1)
        # order by value descending, then id ascending
        order = np.lexsort((cand_i, -cand_v), axis=1)[:, :2]
        top_v = cand_v[rows, order]
        top_i = cand_i[rows, order]
    arg, arg2 = top_i[:, 0], top_i[:, 1]
    w_top = bf16_bits_to_f32(w_bits[arg]).astype(np.float64)
    w_two = bf16_bits_to_f32(w_bits[np.minimum(arg2, V - 1)]).astype(np.float64)
    scale = np.maximum(np.abs(h * w_top).sum(1), np.abs(h * w_two).sum(1))
    return arg.astype(np.int32), top_v[:, 0] - top_v[:, 1], scale
