"""Pins of the draft-tree builder oracle (Alg. 1 + budget pruning, §5.2):
the paper's worked example, special cases that reduce to simpler rules, and
invariants. None of them re-runs the oracle's own loop."""
import json
import os

import numpy as np
import pytest
from scipy.special import softmax

import oracle
from oracle.tree_build import bf16_bits_to_f32, build_tree_one, prune

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "tree_build_narrative.json")


def f32_to_bf16_bits(x):
    """Round-to-nearest-even float32 -> bf16 bit patterns (finite inputs)."""
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return r.astype(np.uint16)


def random_case(seed, B=3, S=4, V=64, H=24, scale=2.0):
    rng = np.random.default_rng(seed)
    logits = (rng.standard_normal((B, S, V)) * scale).astype(np.float32)
    hot = rng.permutation(V)[:H].astype(np.int32)
    table = f32_to_bf16_bits(rng.standard_normal((H, H)) * scale)
    root = rng.integers(0, V, B).astype(np.int32)
    return logits, root, table, hot


# ---------------------------------------------------------------- worked example
def narrative():
    g = json.load(open(GOLDEN))
    vocab = g["vocab"]
    ids = {t: i for i, t in enumerate(vocab)}
    V, S = len(vocab), len(g["steps"])
    logits = np.full((1, S, V), -1e4, dtype=np.float32)
    table = np.zeros((V, V), dtype=np.float32)
    for i, st in enumerate(g["steps"]):
        for t, p in st["logits"].items():
            logits[0, i, ids[t]] = np.float32(np.log(p))
        for row, visible in st["masks"].items():
            table[ids[row]] = g["mask_value"]
            for t in visible:
                table[ids[row], ids[t]] = 0.0
    hot = np.arange(V, dtype=np.int32)
    return g, ids, logits, f32_to_bf16_bits(table), hot


def test_narrative_tree():
    g, ids, logits, table, hot = narrative()
    tok, par, prob, joint = build_tree_one(logits[0], ids[g["root"]], bf16_bits_to_f32(table),
                                           hot, g["k"])
    names = g["vocab"]
    assert len(tok) == len(g["expected_nodes"])
    for n, (t, p_name, jp) in enumerate(g["expected_nodes"]):
        assert names[tok[n]] == t, (n, names[tok[n]], t)
        assert (par[n] < 0) == (p_name is None)
        if p_name is not None:
            assert names[tok[par[n]]] == p_name
        assert joint[n] == pytest.approx(jp, rel=1e-6), (n, t)
    # the printed products
    server = next(n for n in range(len(tok)) if names[tok[n]] == "server")
    assert joint[server] == pytest.approx(0.6 * 0.7, rel=1e-6)
    deep = next(n for n in range(len(tok)) if names[tok[n]] == "optimization" and par[n] == server)
    assert joint[deep] == pytest.approx(0.6 * 0.7 * 0.7, rel=1e-6)
    # frontier after step 2: the two largest joints of that step
    step2 = list(range(3, 7))
    top2 = sorted(step2, key=lambda n: -joint[n])[:2]
    assert [names[tok[n]] for n in top2] == g["expected_frontier_after_step2"]
    # only the frontier nodes have children in step 3
    assert sorted({par[n] for n in range(7, len(tok))}) == sorted(top2)


def test_narrative_budget():
    g, ids, logits, table, hot = narrative()
    par, tok, jnt, nn = oracle.tree_build(logits, np.array([ids[g["root"]]], np.int32), table,
                                          hot, g["k"], 6)
    names = g["vocab"]
    assert nn[0] == 6
    got = []
    for i in range(6):
        label = names[tok[0, i]]
        if label == "optimization":
            label += "@" + names[tok[0, par[0, i]]]
        got.append(label)
    assert got == g["budget_6_keeps"]


# ---------------------------------------------------------------- special cases
def test_k1_is_greedy_decoding_with_token_info():
    """k = 1: the tree is a chain, each token the argmax of l_i plus the
    previous token's table row."""
    logits, root, table, hot = random_case(3, B=4, S=6)
    tab = bf16_bits_to_f32(table)
    hot_index = {int(v): c for c, v in enumerate(hot)}
    par, tok, jnt, nn = oracle.tree_build(logits, root, table, hot, 1, 16)
    for b in range(4):
        assert nn[b] == 7
        prev, jp = int(root[b]), 1.0
        assert tok[b, 0] == prev and par[b, 0] == -1
        for i in range(6):
            x = logits[b, i].copy()
            if prev in hot_index:
                for c, v in enumerate(hot):
                    x[v] = np.float32(x[v] + tab[hot_index[prev], c])
            nxt = int(np.argmax(x))
            jp *= softmax(x.astype(np.float64))[nxt]
            assert tok[b, i + 1] == nxt and par[b, i + 1] == i
            assert jnt[b, i + 1] == pytest.approx(jp, rel=1e-12)
            prev = nxt


def test_no_token_info_gives_identical_sibling_sets():
    """Without hot tokens every frontier node of a step sees the same
    distribution: its children are the top-k of softmax(l_i), with the same
    probabilities."""
    rng = np.random.default_rng(5)
    S, V, k = 4, 40, 3
    logits = rng.standard_normal((1, S, V)).astype(np.float32)
    hot = np.zeros(0, np.int32)
    table = np.zeros((0, 0), np.uint16)
    tok, par, prob, joint = build_tree_one(logits[0], 7, bf16_bits_to_f32(table), hot, k)
    for i in range(S):
        p = softmax(logits[0, i].astype(np.float64))
        want = np.argsort(-p, kind="stable")[:k]
        first = 1 + (0 if i == 0 else k + (i - 1) * k * k)
        n_parents = 1 if i == 0 else k
        for f in range(n_parents):
            kids = range(first + f * k, first + (f + 1) * k)
            assert [tok[n] for n in kids] == list(want)
            assert [prob[n] for n in kids] == pytest.approx(list(p[want]), rel=1e-12)


def test_children_of_full_expansion_sum_to_one():
    """k = V: every expanded node's children are the whole vocabulary and their
    probabilities sum to 1 (the softmax denominator covers hot and non-hot
    tokens alike)."""
    logits, root, table, hot = random_case(11, B=1, S=2, V=9, H=5)
    tok, par, prob, joint = build_tree_one(logits[0], int(root[0]), bf16_bits_to_f32(table),
                                           hot.astype(np.int64), 9)
    par = np.array(par)
    for f in np.unique(par[par >= 0]):
        kids = np.flatnonzero(par == f)
        assert sorted(tok[n] for n in kids) == list(range(9))
        assert sum(prob[n] for n in kids) == pytest.approx(1.0, abs=1e-12)


def test_token_info_row_and_column():
    """A large table entry (row = the node's token, column = a candidate)
    makes that candidate the node's first child; a node whose token is not hot
    gets no token information at all."""
    rng = np.random.default_rng(2)
    V, H = 30, 10
    hot = rng.permutation(V)[:H].astype(np.int32)
    logits = rng.standard_normal((1, 1, V)).astype(np.float32)
    tab = np.zeros((H, H), np.float32)
    tab[4, 7] = 50.0                                   # row hot[4], column hot[7]
    table = f32_to_bf16_bits(tab)
    tok, _, prob, _ = build_tree_one(logits[0], int(hot[4]), bf16_bits_to_f32(table),
                                     hot.astype(np.int64), 2)
    assert tok[1] == hot[7] and prob[1] > 0.99
    tok2, _, _, _ = build_tree_one(logits[0], int(hot[7]), bf16_bits_to_f32(table),
                                   hot.astype(np.int64), 2)
    assert tok2[1] == int(np.argmax(logits[0, 0]))     # row 7 is zero
    non_hot = next(v for v in range(V) if v not in set(hot.tolist()))
    tok3, _, _, _ = build_tree_one(logits[0], non_hot, bf16_bits_to_f32(table),
                                   hot.astype(np.int64), 3)
    assert tok3[1:] == list(np.argsort(-logits[0, 0], kind="stable")[:3])


def test_hot_list_order_does_not_matter():
    """Permuting the hot list together with the table's rows and columns
    leaves the tree unchanged."""
    logits, root, table, hot = random_case(8)
    perm = np.random.default_rng(1).permutation(hot.shape[0])
    a = oracle.tree_build(logits, root, table, hot, 3, 20)
    b = oracle.tree_build(logits, root, table[perm][:, perm], hot[perm], 3, 20)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)


# ---------------------------------------------------------------- invariants
@pytest.mark.parametrize("seed", range(6))
def test_tree_invariants(seed):
    logits, root, table, hot = random_case(20 + seed, B=2, S=5, V=80, H=30)
    k = 2 + seed % 3
    tok, par, prob, joint = build_tree_one(logits[0], int(root[0]), bf16_bits_to_f32(table),
                                           hot.astype(np.int64), k)
    n = len(tok)
    assert n == 1 + k + (5 - 1) * k * k
    for i in range(1, n):
        assert 0 <= par[i] < i
        assert joint[i] == pytest.approx(joint[par[i]] * prob[i], rel=1e-15)
        assert joint[i] <= joint[par[i]]
    # exactly k nodes of each step have children in the next step
    depth = [0] * n
    for i in range(1, n):
        depth[i] = depth[par[i]] + 1
    for d in range(1, 5):
        parents = {par[i] for i in range(n) if depth[i] == d + 1}
        assert len(parents) == k and all(depth[p] == d for p in parents)


@pytest.mark.parametrize("budget", [1, 5, 17, 200])
def test_budget_pruning(budget):
    logits, root, table, hot = random_case(31, B=2, S=4, V=50, H=20)
    k = 3
    par, tok, jnt, nn = oracle.tree_build(logits, root, table, hot, k, budget)
    full = 1 + k + 3 * k * k
    for b in range(2):
        t, p, _, j = build_tree_one(logits[b], int(root[b]), bf16_bits_to_f32(table),
                                    hot.astype(np.int64), k)
        n = min(budget, full)
        assert nn[b] == n
        assert par[b, 0] == -1 and tok[b, 0] == root[b]
        for i in range(1, n):
            assert 0 <= par[b, i] < i
        assert (par[b, n:] == -1).all() and (tok[b, n:] == -1).all() and (jnt[b, n:] == 0).all()
        # every kept joint is at least every dropped one
        kept = sorted(jnt[b, :n].tolist())
        dropped = sorted(set(range(full)) - set(), key=lambda i: -j[i])[n:]
        if dropped:
            assert kept[0] >= max(j[i] for i in dropped)
        assert sorted(j, reverse=True)[:n] == pytest.approx(sorted(kept, reverse=True), rel=0)


# ---------------------------------------------------------------- re-sampling (Alg. 2, §5.3)
def resample_narrative():
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                    "resample_narrative.json")))
    vocab = g["vocab"]
    ids = {t: i for i, t in enumerate(vocab)}
    V, S = len(vocab), len(g["steps"])
    logits = np.full((1, S, V), -1e4, dtype=np.float32)
    table = np.zeros((V, V), dtype=np.float32)
    for i, st in enumerate(g["steps"]):
        for t, p in st["logits"].items():
            logits[0, i, ids[t]] = np.float32(np.log(p))
        for row, visible in st["masks"].items():
            table[ids[row]] = g["mask_value"]
            for t in visible:
                table[ids[row], ids[t]] = 0.0
    return g, ids, logits, f32_to_bf16_bits(table), np.arange(V, dtype=np.int32)


def test_resample_narrative():
    g, ids, logits, table, hot = resample_narrative()
    par, tok, jnt, nn = oracle.resample(logits, np.array([ids[g["bonus"]]], np.int32),
                                        np.array([g["accept_len"]], np.int32), table, hot,
                                        g["k"], g["r"], 16)
    names = g["vocab"]
    assert nn[0] == len(g["expected_nodes"])
    for n, (t, p_name, jp) in enumerate(g["expected_nodes"]):
        assert names[tok[0, n]] == t, (n, names[tok[0, n]], t)
        assert (par[0, n] < 0) == (p_name is None)
        if p_name is not None:
            assert names[tok[0, par[0, n]]] == p_name
        assert jnt[0, n] == pytest.approx(jp, rel=1e-6)


def test_resample_threshold_and_empty():
    """N_remain = S - accept_len; at or below r the new tree is the single
    ground-truth node; a sequence that verified nothing gets no tree."""
    logits, root, table, hot = random_case(44, B=4, S=5)
    bonus = np.array([3, 4, 5, 6], np.int32)
    alen = np.array([0, 3, 4, 6], np.int32)          # N_remain: -, 2, 1, -1
    par, tok, jnt, nn = oracle.resample(logits, bonus, alen, table, hot, 2, 1, 20)
    assert nn.tolist() == [0, 1 + 2 + 4, 1, 1]
    assert (tok[0] == -1).all() and (par[0] == -1).all()
    assert tok[2, 0] == 5 and jnt[2, 0] == 1.0 and (tok[2, 1:] == -1).all()
    assert tok[3, 0] == 6 and par[3, 0] == -1


def test_resample_uses_the_remaining_logits():
    """The re-sampled tree of a sequence with accept_len a is the tree the
    builder draws from logits rows a..S-1 with the bonus token as root."""
    logits, root, table, hot = random_case(45, B=3, S=6)
    bonus = np.array([7, 8, 9], np.int32)
    alen = np.array([1, 2, 4], np.int32)
    got = oracle.resample(logits, bonus, alen, table, hot, 3, 0, 30)
    for b in range(3):
        a = int(alen[b])
        want = oracle.tree_build(logits[b:b + 1, a:], bonus[b:b + 1], table, hot, 3, 30)
        for x, y in zip(got, want):
            np.testing.assert_array_equal(x[b], y[0])
