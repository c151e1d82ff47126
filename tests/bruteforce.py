"""Independent brute-force formulations used to pin the CPU oracle.

Nothing here calls the oracle or the GPU library. Each routine reaches the
same quantity by a different route than the oracle's loops:
  - tree visibility as the reflexive-transitive closure of the child->parent
    relation, by repeated boolean matrix squaring (the oracle walks parent
    links per node);
  - the paged prefix gathered by flat token index with numpy fancy indexing;
  - attention as dense matrix products with a [N, L + N] mask;
  - the accepted path by top-down enumeration of every root-to-node path
    (the oracle does a single topological pass).
"""
from __future__ import annotations

import numpy as np


def widen(bits: np.ndarray) -> np.ndarray:
    """bf16 bits -> float64 (exact)."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def visibility_closure(parent: np.ndarray) -> np.ndarray:
    """R[i, j] = True iff tree node j is node i or one of its ancestors."""
    n = len(parent)
    step = np.eye(n, dtype=np.int64)
    for i, p in enumerate(parent):
        if p >= 0:
            step[i, p] = 1
    reach = step > 0
    while True:
        nxt = (reach.astype(np.int64) @ reach.astype(np.int64)) > 0
        if np.array_equal(nxt, reach):
            return reach
        reach = nxt


def gather_prefix(cache: np.ndarray, page_table_b: np.ndarray, L: int) -> np.ndarray:
    """[L, Hkv, D] prefix rows of one sequence from a [pages, P, Hkv, D] cache."""
    P = cache.shape[1]
    flat = cache.reshape(-1, *cache.shape[2:])
    t = np.arange(L)
    return flat[page_table_b[t // P].astype(np.int64) * P + t % P]


def tree_attention_dense(q, k_tree, v_tree, k_cache, v_cache, page_table, kv_len, parent,
                         scale=None):
    q = widen(q)
    kt, vt = widen(k_tree), widen(v_tree)
    B, N, Hq, D = q.shape
    Hkv = kt.shape[2]
    G = Hq // Hkv
    if scale is None or scale <= 0:
        scale = 1.0 / np.sqrt(D)
    out = np.zeros((B, N, Hq, D))
    lse = np.zeros((B, N, Hq))
    for b in range(B):
        L = int(kv_len[b])
        kp = widen(gather_prefix(k_cache, page_table[b], L))
        vp = widen(gather_prefix(v_cache, page_table[b], L))
        mask = np.concatenate([np.ones((N, L), dtype=bool), visibility_closure(parent[b])], axis=1)
        for h in range(Hq):
            g = h // G
            keys = np.concatenate([kp[:, g, :], kt[b, :, g, :]], axis=0)
            vals = np.concatenate([vp[:, g, :], vt[b, :, g, :]], axis=0)
            s = scale * (q[b, :, h, :] @ keys.T)
            s = np.where(mask, s, -np.inf)
            mx = s.max(axis=1, keepdims=True)
            w = np.exp(s - mx)
            den = w.sum(axis=1, keepdims=True)
            out[b, :, h, :] = (w @ vals) / den
            lse[b, :, h] = (mx + np.log(den))[:, 0]
    return out, lse


def children_lists(parent):
    ch = {i: [] for i in range(len(parent))}
    for i, p in enumerate(parent):
        if p >= 0:
            ch[int(p)].append(i)
    return ch


def accept_enumerate(draft, parent, amax):
    """Top-down enumeration of every root-to-node path; keep those whose every
    edge matches (child token == target argmax at the parent); the longest
    wins, ties to the lower terminal index."""
    ch = children_lists(parent)
    paths = []

    def walk(path):
        paths.append(list(path))
        for c in ch[path[-1]]:
            walk(path + [c])

    for r in range(len(parent)):
        if parent[r] < 0:
            walk([r])
    ok = [p for p in paths
          if all(draft[p[k + 1]] == amax[p[k]] for k in range(len(p) - 1))]
    best = min(ok, key=lambda p: (-len(p), p[-1]))
    return len(best), best, int(amax[best[-1]])


def compact_scatter(k_tree, v_tree, k_cache, v_cache, page_table, kv_len, accept_idx, accept_len):
    kc = k_cache.copy()
    vc = v_cache.copy()
    P = kc.shape[1]
    fk = kc.reshape(-1, *kc.shape[2:])
    fv = vc.reshape(-1, *vc.shape[2:])
    for b in range(len(kv_len)):
        n = int(accept_len[b])
        pos = int(kv_len[b]) + np.arange(n)
        dst = page_table[b][pos // P].astype(np.int64) * P + pos % P
        src = accept_idx[b, :n]
        fk[dst] = k_tree[b, src]
        fv[dst] = v_tree[b, src]
    return kc, vc
