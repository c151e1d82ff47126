"""Oracle of the draft-tree builder: token-info sampling (Alg. 1) followed by
the verification-budget pruning (§5.2). TEST INFRASTRUCTURE ONLY, like the
rest of this package: plain numpy, fp64 probabilities, one node at a time.

What is computed, per sequence (the steps follow Alg. 1 in the paper's order):

* The root is the last verified token, with probability and joint
  probability 1, and forms the first frontier.
* Step i (1..S) uses the draft logits l_i. For every frontier node, in
  frontier order, the node's token-info row is added to l_i (§5.1: the
  collapsed token-info embedding is an additive logit table), the sum is
  normalised by a softmax, and the k most probable tokens become the node's
  children, in rank order, each with its probability p and the joint
  probability parent.joint * p.
* The next frontier is the k children of this step with the largest joint
  probabilities, largest first (not all k*k of them: the tree does not grow
  exponentially); the next step expands them in that order.
* After the last step the tree is pruned to the verification budget: the
  `budget` nodes with the largest joint probabilities are kept (§5.2).

Readings where the paper is silent (each one is also a row of the design
notes):

* What a table entry is: §4.1 adds RMSNorm(E'(t)) to the logits of the step
  after token t, §5.1 collapses E' into a lookup table and says sampling does
  no further computation on it, so a stored row is taken to be the already
  normalised vector RMSNorm(E'(t)) (the normalisation of a fixed row is a
  constant, computed offline over the whole row). Entry (row, col) is that
  vector's component for candidate col, added to the logit as it is.
* The token-info table only covers the hot tokens (§6.1 keeps token-info for
  the 32K most frequent tokens only): `table` is [H, H] over the hot list
  `hot`, row = the node's token, column = the candidate token, i.e. the
  normalised rows above restricted to hot rows and hot columns. A node whose
  token is not hot adds nothing; a candidate that is not hot gets nothing
  added. Table entries are bf16; the sum l + r is formed in fp32, the precision
  of the logits, and top-k decisions are taken on these fp32 sums.
* Ties: equal sums rank the lower vocabulary id first; equal joint
  probabilities rank the node created first (creation order = step, then
  frontier rank, then child rank). A child's joint probability never exceeds
  its parent's, so the kept set always contains the parents of its nodes.
* Output order is creation order restricted to the kept nodes: node 0 is the
  root, every parent precedes its children, and a tree smaller than the budget
  leaves padding slots (parent -1, token -1, joint 0).
"""
from __future__ import annotations

import numpy as np


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) to the float32 values they denote."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _topk_by_value(x: np.ndarray, k: int) -> np.ndarray:
    """Indices of the k largest entries of x, larger value first, lower index on ties."""
    order = np.lexsort((np.arange(x.shape[0]), -x.astype(np.float64)))
    return order[:k]


def build_tree_one(logits: np.ndarray, root: int, table: np.ndarray, hot: np.ndarray, k: int,
                   margins: list | None = None):
    """Alg. 1 for one sequence without pruning.

    logits [S, V] float32, root token id, table [H, H] float32 (bf16 values)
    or uint16 (bf16 bit patterns, converted one row at a time), hot [H] vocab ids. Returns parallel lists (token, parent, prob, joint) in
    creation order. When `margins` is a list, the relative gap between the
    last frontier node kept and the first one dropped is appended per step.
    """
    S, V = logits.shape
    hot_index = np.full(V, -1, dtype=np.int64)
    hot_index[hot] = np.arange(hot.shape[0])
    token, parent, prob, joint = [int(root)], [-1], [1.0], [1.0]
    frontier = [0]
    for i in range(S):
        l_i = logits[i].astype(np.float32)
        children = []
        for f in frontier:
            x = l_i.copy()
            h = hot_index[token[f]]
            if h >= 0:
                row = table[h]
                if row.dtype == np.uint16:
                    row = bf16_bits_to_f32(row)
                x[hot] = (l_i[hot] + row).astype(np.float32)
            x64 = x.astype(np.float64)
            m = x64.max()
            s = np.exp(x64 - m).sum()
            for e in _topk_by_value(x, k):
                p = float(np.exp(x64[e] - m) / s)
                token.append(int(e))
                parent.append(f)
                prob.append(p)
                joint.append(joint[f] * p)
                children.append(len(token) - 1)
        ranked = sorted(children, key=lambda n: (-joint[n], n))
        if margins is not None and len(ranked) > k:
            a, b = joint[ranked[k - 1]], joint[ranked[k]]
            margins.append((a - b) / a if a > 0 else 0.0)
        frontier = ranked[:k]
    return token, parent, prob, joint


def prune(token, parent, joint, budget: int):
    """The `budget` nodes of largest joint probability, in creation order, with
    parents renumbered. Returns (parent, token, joint, n) arrays of length budget."""
    n_all = len(token)
    keep = sorted(sorted(range(n_all), key=lambda n: (-joint[n], n))[:budget])
    new = {old: i for i, old in enumerate(keep)}
    out_p = np.full(budget, -1, dtype=np.int32)
    out_t = np.full(budget, -1, dtype=np.int32)
    out_j = np.zeros(budget, dtype=np.float64)
    for i, old in enumerate(keep):
        out_t[i] = token[old]
        out_j[i] = joint[old]
        out_p[i] = -1 if parent[old] < 0 else new[parent[old]]
    return out_p, out_t, out_j, len(keep)


def tree_build(logits, root, table_bits, hot, k: int, budget: int, margins: list | None = None):
    """Alg. 1 + budget pruning for a batch.

    logits [B, S, V] float32; root [B] int32; table_bits [H, H] uint16 (bf16);
    hot [H] int32 distinct vocab ids. Returns parent [B, budget] int32, token
    [B, budget] int32, joint [B, budget] float64 and num_nodes [B] int32. With a
    `margins` list, the relative gap at every frontier choice and at the
    pruning cut is appended (how close the decision was to a tie).
    """
    logits = np.asarray(logits, dtype=np.float32)
    B = logits.shape[0]
    table = np.asarray(table_bits, dtype=np.uint16)
    hot = np.asarray(hot, dtype=np.int64)
    par = np.full((B, budget), -1, dtype=np.int32)
    tok = np.full((B, budget), -1, dtype=np.int32)
    jnt = np.zeros((B, budget), dtype=np.float64)
    nn = np.zeros(B, dtype=np.int32)
    for b in range(B):
        t, p, _, j = build_tree_one(logits[b], int(root[b]), table, hot, k, margins)
        if margins is not None and len(j) > budget:
            js = sorted(j, reverse=True)
            margins.append((js[budget - 1] - js[budget]) / js[budget - 1])
        par[b], tok[b], jnt[b], nn[b] = prune(t, p, j, budget)
    return par, tok, jnt, nn


def resample(logits, bonus, accept_len, table_bits, hot, k: int, r: int, budget: int,
             margins: list | None = None):
    """Re-sampling (Alg. 2, §5.3) for a batch after verification.

    The ground-truth token is the verification's bonus token; the first
    rejected draft position is accept_len (the accepted path counts the root at
    depth 0, so the token at depth accept_len was rejected and was drawn from
    logits row accept_len - 1). The remaining logits are rows accept_len ..
    S-1 and N_remain = S - accept_len. If N_remain > r the new tree is
    BuildSubtree(remaining logits, bonus, k, N_remain), pruned to the budget
    like a first tree; otherwise it is the single ground-truth node. A sequence
    that verified nothing (accept_len 0) gets an empty tree.
    Returns parent, token, joint, num_nodes as tree_build does.
    """
    logits = np.asarray(logits, dtype=np.float32)
    B, S, _ = logits.shape
    table = np.asarray(table_bits, dtype=np.uint16)
    hot = np.asarray(hot, dtype=np.int64)
    par = np.full((B, budget), -1, dtype=np.int32)
    tok = np.full((B, budget), -1, dtype=np.int32)
    jnt = np.zeros((B, budget), dtype=np.float64)
    nn = np.zeros(B, dtype=np.int32)
    for b in range(B):
        a = int(accept_len[b])
        if a <= 0:
            continue
        n_remain = S - a
        if n_remain > r:
            t, p, _, j = build_tree_one(logits[b, a:], int(bonus[b]), table, hot, k, margins)
            if margins is not None and len(j) > budget:
                js = sorted(j, reverse=True)
                margins.append((js[budget - 1] - js[budget]) / js[budget - 1])
            par[b], tok[b], jnt[b], nn[b] = prune(t, p, j, budget)
        else:
            tok[b, 0], jnt[b, 0], nn[b] = int(bonus[b]), 1.0, 1
    return par, tok, jnt, nn

