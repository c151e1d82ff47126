"""Pins for the oracle's tree attention (CPU only).

Each test reaches the expected value by a route the oracle does not take: a
dense brute force over the closure of the parent relation, the CPU library's
scaled-dot-product attention for the shapes where a tree reduces to textbook
attention (a chain is causal attention; a single node is decode attention),
closed forms, and invariances the definition implies (§2.1 tree-shaped
verification mask; §8 SpecInfer masking; §1 attention over the KV cache).
"""
import math

import numpy as np
import pytest
import torch

from paper_2602_21224_amd import workloads as W
from tests import bruteforce as BF

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def small(seed, *, B=2, N=7, Hq=4, Hkv=2, D=8, L=(0, 40), P=4, tree="forest", poison=False):
    if tree == "forest":
        fn = lambda r: W.tree_uniform_forest(r, N)
    elif tree == "chain":
        fn = lambda r: W.tree_chain(N)
    elif tree == "star":
        fn = lambda r: W.tree_star(N)
    else:
        fn = lambda r: W.tree_random_depth_capped(r, N, 3)
    return W.make_workload("t", seed, B=B, N=N, Hq=Hq, Hkv=Hkv, D=D, kv_len=L, parent_fn=fn,
                           V=50, P=P, poison=poison, with_logits=False)


def run(oracle_mod, w, scale=0.0, **over):
    a = dict(q=w.q, k_tree=w.k_tree, v_tree=w.v_tree, k_cache=w.k_cache, v_cache=w.v_cache,
             page_table=w.page_table, kv_len=w.kv_len, parent=w.parent)
    a.update(over)
    return oracle_mod.tree_attention(**a, scale=scale)


CASES = []
for N in (1, 2, 5, 12):
    for L in (0, 1, 15, 16, 17, 40):
        for D, G, P in ((8, 1, 1), (8, 2, 4), (64, 4, 16)):
            CASES.append((N, L, D, G, P))


@pytest.mark.parametrize("N,L,D,G,P", CASES)
def test_matches_dense_bruteforce(oracle_mod, N, L, D, G, P):
    w = small(1000 * N + 10 * L + D + G + P, B=2, N=N, Hq=2 * G, Hkv=2, D=D, L=L, P=P,
              poison=True)
    out, lse = run(oracle_mod, w)
    ref, rlse = BF.tree_attention_dense(w.q, w.k_tree, w.v_tree, w.k_cache, w.v_cache,
                                        w.page_table, w.kv_len, w.parent)
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(lse, rlse, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("tree", ["forest", "capped", "star"])
def test_random_trees_ragged_lengths(oracle_mod, tree):
    w = small(7, B=3, N=12, Hq=8, Hkv=2, D=16, L=(0, 50), P=16, tree=tree, poison=True)
    out, lse = run(oracle_mod, w, scale=0.37)
    ref, rlse = BF.tree_attention_dense(w.q, w.k_tree, w.v_tree, w.k_cache, w.v_cache,
                                        w.page_table, w.kv_len, w.parent, scale=0.37)
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(lse, rlse, rtol=1e-12, atol=1e-12)


def _sdpa(qv, keys, vals, mask, scale):
    """CPU library attention in float64; qv [Hq, M, D], keys/vals [Hq, S, D]."""
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a))
    o = torch.nn.functional.scaled_dot_product_attention(
        t(qv), t(keys), t(vals), attn_mask=None if mask is None else t(mask), scale=scale)
    return o.numpy()


@pytest.mark.parametrize("L,N,G", [(0, 9, 1), (23, 9, 2), (40, 16, 4)])
def test_chain_equals_causal_attention(oracle_mod, L, N, G):
    """A chain-shaped tree is ordinary causal attention over [prefix; chain]."""
    w = small(11 + L, B=1, N=N, Hq=2 * G, Hkv=2, D=32, L=L, P=4, tree="chain")
    out, _ = run(oracle_mod, w)
    q = BF.widen(w.q[0]).transpose(1, 0, 2)                       # [Hq, N, D]
    kp = BF.widen(BF.gather_prefix(w.k_cache, w.page_table[0], L))
    vp = BF.widen(BF.gather_prefix(w.v_cache, w.page_table[0], L))
    keys = np.concatenate([kp, BF.widen(w.k_tree[0])], axis=0)    # [L+N, Hkv, D]
    vals = np.concatenate([vp, BF.widen(w.v_tree[0])], axis=0)
    keys = np.repeat(keys, G, axis=1).transpose(1, 0, 2)          # [Hq, L+N, D]
    vals = np.repeat(vals, G, axis=1).transpose(1, 0, 2)
    mask = np.tril(np.ones((N, L + N), dtype=bool), k=L)          # causal, prefix visible
    ref = _sdpa(q, keys, vals, mask, 1.0 / math.sqrt(32))
    np.testing.assert_allclose(out[0].transpose(1, 0, 2), ref, rtol=1e-10, atol=1e-12)


@pytest.mark.parametrize("L", [0, 1, 37, 128])
def test_single_node_equals_decode_attention(oracle_mod, L):
    """N = 1: every head is plain decode attention over the prefix plus itself."""
    w = small(5 + L, B=2, N=1, Hq=8, Hkv=2, D=64, L=L, P=16)
    out, _ = run(oracle_mod, w)
    for b in range(2):
        q = BF.widen(w.q[b]).transpose(1, 0, 2)                   # [Hq, 1, D]
        kp = BF.widen(BF.gather_prefix(w.k_cache, w.page_table[b], L))
        vp = BF.widen(BF.gather_prefix(w.v_cache, w.page_table[b], L))
        keys = np.repeat(np.concatenate([kp, BF.widen(w.k_tree[b])]), 4, axis=1).transpose(1, 0, 2)
        vals = np.repeat(np.concatenate([vp, BF.widen(w.v_tree[b])]), 4, axis=1).transpose(1, 0, 2)
        ref = _sdpa(q, keys, vals, None, 1.0 / 8.0)
        np.testing.assert_allclose(out[b].transpose(1, 0, 2), ref, rtol=1e-10, atol=1e-12)


def test_single_node_empty_prefix_closed_form(oracle_mod):
    """N = 1 and L = 0: the only visible key is the node itself, so the output
    is its value row and the log-sum-exp is its own scaled score."""
    w = small(3, B=3, N=1, Hq=4, Hkv=4, D=64, L=0, P=16)
    out, lse = run(oracle_mod, w, scale=0.25)
    np.testing.assert_array_equal(out, BF.widen(w.v_tree))
    qk = (BF.widen(w.q) * BF.widen(w.k_tree)).sum(-1) * 0.25
    np.testing.assert_allclose(lse, qk, rtol=1e-14, atol=1e-14)


def test_hand_worked_example(oracle_mod):
    """Two prefix keys, tree 0 <- {1, 2}; node 2 sees p0, p1, t0, t2 (not t1).
    Scores with scale 1: 0, 1, 0, 2, so the weights are 1, e, 1, e^2."""
    bf = W.f32_to_bf16_bits
    k_cache = bf(np.array([[[[0, 0]]], [[[1, 0]]]], np.float32))   # pages of P=1
    v_cache = bf(np.array([[[[1, 0]]], [[[0, 1]]]], np.float32))
    k_tree = bf(np.array([[[[0, 0]], [[5, 5]], [[2, 0]]]], np.float32))
    v_tree = bf(np.array([[[[0, 0]], [[100, 100]], [[1, 1]]]], np.float32))
    q = bf(np.array([[[[1, 0]], [[1, 0]], [[1, 0]]]], np.float32))
    page_table = np.array([[0, 1, -1, -1, -1]], np.int32)
    out, lse = oracle_mod.tree_attention(q, k_tree, v_tree, k_cache, v_cache, page_table,
                                         np.array([2], np.int32),
                                         np.array([[-1, 0, 0]], np.int32), scale=1.0)
    e = math.e
    den = 2 + e + e * e
    np.testing.assert_allclose(out[0, 2, 0], [(1 + e * e) / den, (e + e * e) / den], rtol=1e-15)
    np.testing.assert_allclose(lse[0, 2, 0], math.log(den), rtol=1e-15)
    # node 0 sees p0, p1, t0 with scores 0, 1, 0
    np.testing.assert_allclose(out[0, 0, 0], [1 / (2 + e), e / (2 + e)], rtol=1e-15)


def test_constant_values_give_that_constant(oracle_mod):
    w = small(21, B=2, N=10, Hq=4, Hkv=2, D=16, L=(3, 30), P=4)
    c = W.f32_to_bf16_bits(np.linspace(-2, 2, 16, dtype=np.float32))
    vc = np.broadcast_to(c, w.v_cache.shape).copy()
    vt = np.broadcast_to(c, w.v_tree.shape).copy()
    out, _ = run(oracle_mod, w, v_cache=vc, v_tree=vt)
    np.testing.assert_allclose(out, np.broadcast_to(BF.widen(c), out.shape), rtol=1e-13,
                               atol=1e-13)


def test_identical_keys_give_mean_of_visible_values(oracle_mod):
    """Equal scores: the output is the plain mean over the L prefix rows and the
    node's root path (depth + 1 rows)."""
    w = small(22, B=2, N=10, Hq=4, Hkv=2, D=16, L=(3, 30), P=4)
    k = W.f32_to_bf16_bits(np.full(16, 0.5, np.float32))
    out, _ = run(oracle_mod, w, k_cache=np.broadcast_to(k, w.k_cache.shape).copy(),
                 k_tree=np.broadcast_to(k, w.k_tree.shape).copy())
    for b in range(2):
        L = int(w.kv_len[b])
        vp = BF.widen(BF.gather_prefix(w.v_cache, w.page_table[b], L))
        for i in range(10):
            path = [i]
            while w.parent[b, path[-1]] >= 0:
                path.append(int(w.parent[b, path[-1]]))
            rows = np.concatenate([vp, BF.widen(w.v_tree[b, path])])     # [L+len, Hkv, D]
            mean = rows.mean(axis=0)
            for h in range(4):
                np.testing.assert_allclose(out[b, i, h], mean[h // 2], rtol=1e-12, atol=1e-12)


def test_page_permutation_is_invisible(oracle_mod):
    w = small(31, B=3, N=8, Hq=4, Hkv=2, D=16, L=(5, 60), P=4)
    out, lse = run(oracle_mod, w)
    rng = np.random.default_rng(9)
    perm = rng.permutation(w.num_pages)              # new physical slot of each page
    kc = np.empty_like(w.k_cache)
    vc = np.empty_like(w.v_cache)
    kc[perm] = w.k_cache
    vc[perm] = w.v_cache
    pt = np.where(w.page_table >= 0, perm[np.maximum(w.page_table, 0)], -1).astype(np.int32)
    out2, lse2 = run(oracle_mod, w, k_cache=kc, v_cache=vc, page_table=pt)
    np.testing.assert_array_equal(out, out2)
    np.testing.assert_array_equal(lse, lse2)


def test_invisible_rows_do_not_matter(oracle_mod):
    """Poisoning cache slots past each prefix with NaN, and tree rows that are
    not on a node's root path with +-1e4, leaves that node's output unchanged."""
    w = small(41, B=2, N=12, Hq=4, Hkv=2, D=16, L=(1, 40), P=4)
    out, lse = run(oracle_mod, w)
    kc, vc = w.k_cache.copy(), w.v_cache.copy()
    W.poison_cache_tails(kc, vc, w.page_table, w.kv_len, w.P)
    out_p, lse_p = run(oracle_mod, w, k_cache=kc, v_cache=vc)
    np.testing.assert_array_equal(out, out_p)
    np.testing.assert_array_equal(lse, lse_p)
    big = W.f32_to_bf16_bits(np.float32(1e4))
    for b in range(2):
        vis = BF.visibility_closure(w.parent[b])
        for i in range(12):
            kt, vt = w.k_tree.copy(), w.v_tree.copy()
            hide = ~vis[i]
            kt[b, hide] = big
            vt[b, hide] = big ^ np.uint16(0x8000)
            o2, l2 = run(oracle_mod, w, k_tree=kt, v_tree=vt)
            np.testing.assert_array_equal(out[b, i], o2[b, i])
            np.testing.assert_array_equal(lse[b, i], l2[b, i])


def test_gqa_equals_expanded_mha(oracle_mod):
    """Query head h reads KV head h // G: duplicating each KV head G times and
    running multi-head attention gives identical results."""
    G = 4
    w = small(51, B=2, N=9, Hq=8, Hkv=2, D=16, L=(4, 33), P=4)
    out, lse = run(oracle_mod, w)
    rep = lambda a: np.repeat(a, G, axis=2)
    out2, lse2 = run(oracle_mod, w, k_tree=rep(w.k_tree), v_tree=rep(w.v_tree),
                     k_cache=rep(w.k_cache), v_cache=rep(w.v_cache))
    np.testing.assert_array_equal(out, out2)
    np.testing.assert_array_equal(lse, lse2)


def test_default_scale_is_inverse_sqrt_head_dim(oracle_mod):
    w = small(61, B=1, N=6, Hq=2, Hkv=1, D=64, L=20, P=4)
    a, la = run(oracle_mod, w, scale=0.0)
    b, lb = run(oracle_mod, w, scale=0.125)
    np.testing.assert_array_equal(a, b)
    np.testing.assert_array_equal(la, lb)


def test_rejects_malformed_tree(oracle_mod):
    w = small(71, B=1, N=4, Hq=2, Hkv=1, D=8, L=4, P=4)
    bad = w.parent.copy()
    bad[0, 2] = 2
    with pytest.raises(ValueError):
        run(oracle_mod, w, parent=bad)


def test_rows_entry_matches_full(oracle_mod):
    w = small(81, B=3, N=11, Hq=8, Hkv=2, D=32, L=(0, 45), P=4, poison=True)
    out, lse = run(oracle_mod, w)
    rng = np.random.default_rng(0)
    items = np.stack([rng.integers(0, 3, 40), rng.integers(0, 11, 40), rng.integers(0, 8, 40)], 1)
    o2, l2 = oracle_mod.tree_attention_rows(w.q, w.k_tree, w.v_tree, w.k_cache, w.v_cache,
                                            w.page_table, w.kv_len, w.parent, items)
    np.testing.assert_array_equal(o2, out[items[:, 0], items[:, 1], items[:, 2]])
    np.testing.assert_array_equal(l2, lse[items[:, 0], items[:, 1], items[:, 2]])
