"""Seeded synthetic inputs for the target-model tree-verification step.

This module only *draws* inputs: draft trees (parent links and token ids), a
paged bf16 KV cache, bf16 queries and tree keys/values, and fp32 vocabulary
logits. It performs none of the verification arithmetic (no attention, no
argmax, no acceptance, no compaction), so both the GPU path and the CPU oracle
can consume the same bytes without sharing any of the method's code.

Shapes follow the draft-tree verification setting of the paper: a tree of
draft tokens whose nodes carry a token and a parent (Alg. 1's Node structure,
§5.2), rooted at the last verified token (§5.2), verified in one target pass
over a paged KV cache (§7.1 uses Paged Attention). The five named presets are
Llama-shaped stand-ins for the paper's serving workload (§7.1, which uses an
unnamed SGLang benchmark set); no dataset item is reproduced.

Layouts (all C-contiguous):
  q        uint16 (bf16 bits) [B, N, Hq, D]
  k_tree   uint16             [B, N, Hkv, D]
  v_tree   uint16             [B, N, Hkv, D]
  k_cache  uint16             [num_pages, P, Hkv, D]
  v_cache  uint16             [num_pages, P, Hkv, D]
  page_table int32            [B, max_pages]   (-1 beyond what a sequence owns)
  kv_len   int32              [B]
  parent   int32              [B, N]           (parent[b, i] in [-1, i-1])
  draft    int32              [B, N]
  logits   float32            [B, N, V]
  num_nodes int32             [B] or None      (ragged forests: nodes past
                                                num_nodes[b] are padding)
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

PAGE_SIZE = 16
BF16_NAN = np.uint16(0x7FC0)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round finite float32 values to bf16 (round-to-nearest-even), return raw bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounding = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + rounding) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(h: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bits to float32 (used by tests for fixtures)."""
    return (np.asarray(h, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclass
class Workload:
    name: str
    B: int
    N: int
    Hq: int
    Hkv: int
    D: int
    P: int
    V: int
    q: np.ndarray
    k_tree: np.ndarray
    v_tree: np.ndarray
    k_cache: np.ndarray
    v_cache: np.ndarray
    page_table: np.ndarray
    kv_len: np.ndarray
    parent: np.ndarray
    draft: np.ndarray
    logits: np.ndarray | None
    meta: dict = field(default_factory=dict)
    num_nodes: np.ndarray | None = None

    @property
    def max_pages(self) -> int:
        return int(self.page_table.shape[1])

    @property
    def num_pages(self) -> int:
        return int(self.k_cache.shape[0])

    @property
    def max_kv_len(self) -> int:
        return int(self.kv_len.max()) if self.B else 0


# --------------------------------------------------------------------------
# tree shapes (parent arrays in topological order: parent[i] < i)
# --------------------------------------------------------------------------

def tree_uniform_forest(rng: np.random.Generator, n: int) -> np.ndarray:
    """parent[i] uniform over {-1, 0, ..., i-1}; several roots are possible."""
    parent = np.empty(n, dtype=np.int32)
    for i in range(n):
        parent[i] = rng.integers(-1, i) if i > 0 else -1
    return parent


def tree_random_depth_capped(rng: np.random.Generator, n: int, depth_lt: int,
                             root_children: int = 0) -> np.ndarray:
    """Node 0 is the root; optionally nodes 1..root_children hang off it; every
    later node picks a parent uniformly among earlier nodes of depth < depth_lt."""
    parent = np.full(n, -1, dtype=np.int32)
    depth = np.zeros(n, dtype=np.int64)
    for i in range(1, n):
        if i <= root_children:
            p = 0
        else:
            cand = np.nonzero(depth[:i] < depth_lt)[0]
            p = int(cand[rng.integers(0, len(cand))])
        parent[i] = p
        depth[i] = depth[p] + 1
    return parent


def tree_topk_expansion(rng: np.random.Generator, branching, keep: int):
    """Expand a root level by level with the given children-per-node counts;
    child probabilities are the top-b entries of a sorted Dirichlet(1 x 8)
    draw; keep the `keep` nodes of highest joint probability (ties to the
    lower BFS index) and relabel them in BFS order. Returns the parent array.
    This mirrors how a draft tree is built and pruned to a verification budget
    (Alg. 1 and the budget pruning of §5.2) only to shape the synthetic input."""
    par = [-1]
    joint = [1.0]
    frontier = [0]
    for b in branching:
        nxt = []
        for node in frontier:
            probs = np.sort(rng.dirichlet(np.ones(8)))[::-1][:b]
            for pr in probs:
                par.append(node)
                joint.append(joint[node] * float(pr))
                nxt.append(len(par) - 1)
        frontier = nxt
    joint_a = np.asarray(joint)
    order = sorted(range(len(par)), key=lambda i: (-joint_a[i], i))
    kept = sorted(order[:keep])
    relabel = {old: new for new, old in enumerate(kept)}
    parent = np.empty(len(kept), dtype=np.int32)
    for new, old in enumerate(kept):
        p = par[old]
        if p >= 0 and p not in relabel:
            raise AssertionError("pruned tree is not ancestor-closed")
        parent[new] = -1 if p < 0 else relabel[p]
    return parent


def tree_frontier_expansion(rng: np.random.Generator, k: int, steps: int, keep: int):
    """A draft tree the way the paper's evaluation verifies them (§7.1: trees
    of depth 3 at most 4 wide): from the root, each of `steps` levels offers k
    children to every frontier node (probabilities: the top-k entries of a
    sorted Dirichlet(1 x 8) draw), and the k children of largest joint
    probability form the next frontier. The root and the frontier nodes of
    every level make an ancestor-closed tree at most k wide; the `keep` of
    largest joint probability (ties to the node created first) are kept, in
    creation order. Only shapes the synthetic input; returns the parent array."""
    par = [-1]
    joint = [1.0]
    frontier = [0]
    members = [0]
    for _ in range(steps):
        cand = []
        for node in frontier:
            for pr in np.sort(rng.dirichlet(np.ones(8)))[::-1][:k]:
                par.append(node)
                joint.append(joint[node] * float(pr))
                cand.append(len(par) - 1)
        frontier = sorted(cand, key=lambda i: (-joint[i], i))[:k]
        members += sorted(frontier)
    kept = sorted(sorted(members, key=lambda i: (-joint[i], i))[:keep])
    relabel = {old: new for new, old in enumerate(kept)}
    parent = np.empty(len(kept), dtype=np.int32)
    for new, old in enumerate(kept):
        p = par[old]
        if p >= 0 and p not in relabel:
            raise AssertionError("pruned tree is not ancestor-closed")
        parent[new] = -1 if p < 0 else relabel[p]
    return parent


def fusion_forest(rng: np.random.Generator, primary, resampled, depth_lt: int) -> np.ndarray:
    """Input of a fused verification (§6.2: the previous round's re-sampled
    trees are verified together with the next batch): this round's draft tree
    (root 0) followed by a re-sampled tree with its own root (Alg. 2 roots it
    at the ground-truth token). `primary` and `resampled` are inclusive node
    count ranges; both trees are depth-capped random trees."""
    n1 = int(rng.integers(primary[0], primary[1] + 1))
    n2 = int(rng.integers(resampled[0], resampled[1] + 1))
    a = tree_random_depth_capped(rng, n1, depth_lt)
    if n2 == 0:
        return a
    c = tree_random_depth_capped(rng, n2, depth_lt)
    c = np.where(c >= 0, c + n1, -1).astype(np.int32)
    return np.concatenate([a, c]).astype(np.int32)


def tree_depths(parent: np.ndarray) -> np.ndarray:
    d = np.zeros(len(parent), dtype=np.int64)
    for i, p in enumerate(parent):
        d[i] = 0 if p < 0 else d[p] + 1
    return d


def tree_chain(n: int) -> np.ndarray:
    return np.arange(-1, n - 1, dtype=np.int32)


def tree_star(n: int) -> np.ndarray:
    p = np.zeros(n, dtype=np.int32)
    p[0] = -1
    return p


# --------------------------------------------------------------------------
# draft tokens and logits
# --------------------------------------------------------------------------

def draft_tokens(rng: np.random.Generator, parent: np.ndarray, V: int,
                 distinct_siblings: bool) -> np.ndarray:
    n = len(parent)
    tok = rng.integers(0, V, size=n).astype(np.int32)
    if distinct_siblings:
        seen: dict[int, set] = {}
        for i in range(n):
            s = seen.setdefault(int(parent[i]), set())
            while int(tok[i]) in s and len(s) < V:
                tok[i] = rng.integers(0, V)
            s.add(int(tok[i]))
    return tok


def boost_logits(rng: np.random.Generator, logits_b: np.ndarray, parent: np.ndarray,
                 draft: np.ndarray, prob: float, amount: float) -> None:
    """For each node that has children, with probability `prob` add `amount`
    to that node's logit of one uniformly chosen child's draft token."""
    n = len(parent)
    children: dict[int, list] = {}
    for i in range(n):
        if parent[i] >= 0:
            children.setdefault(int(parent[i]), []).append(i)
    for p in range(n):
        ch = children.get(p)
        if not ch:
            continue
        if rng.random() < prob:
            c = ch[int(rng.integers(0, len(ch)))]
            logits_b[p, draft[c]] += np.float32(amount)


# --------------------------------------------------------------------------
# paged cache
# --------------------------------------------------------------------------

def paged_layout(rng: np.random.Generator, kv_len: np.ndarray, N: int, P: int):
    """Give each sequence ceil((L_b + N) / P) pages (room for the accepted
    path), drawn from one seeded permutation of the pool. Returns
    (page_table [B, max_pages] with -1 padding, num_pages)."""
    need = [(int(L) + N + P - 1) // P for L in kv_len]
    total = int(sum(need))
    max_pages = max(need) if need else 1
    perm = rng.permutation(total).astype(np.int32)
    pt = np.full((len(kv_len), max_pages), -1, dtype=np.int32)
    off = 0
    for b, k in enumerate(need):
        pt[b, :k] = perm[off:off + k]
        off += k
    return pt, total


def _normal_bf16(rng: np.random.Generator, shape) -> np.ndarray:
    return f32_to_bf16_bits(rng.standard_normal(size=shape, dtype=np.float32))


def poison_cache_tails(k_cache, v_cache, page_table, kv_len, P) -> None:
    """Fill every cache slot that no sequence's prefix covers with bf16 NaN."""
    num_pages = k_cache.shape[0]
    used = np.zeros((num_pages, P), dtype=bool)
    for b in range(len(kv_len)):
        L = int(kv_len[b])
        for t in range(0, L, P):
            pg = page_table[b, t // P]
            used[pg, : min(P, L - t)] = True
    k_cache[~used] = BF16_NAN
    v_cache[~used] = BF16_NAN


def make_workload(name: str, seed: int, *, B: int, N: int, Hq: int, Hkv: int, D: int,
                  kv_len, parent_fn, V: int, boost_prob: float = 0.0,
                  boost_amount: float = 3.0, P: int = PAGE_SIZE,
                  distinct_siblings: bool = True, poison: bool = False,
                  with_logits: bool = True, forced_path=None) -> Workload:
    """Draw one workload. `kv_len` is an int, a (lo, hi) inclusive range, or
    an explicit per-sequence list; `parent_fn(rng)` returns one tree of at most
    N nodes. If any tree is shorter than N the batch is ragged: `num_nodes`
    holds each sequence's node count and every input row of the padding nodes
    is poisoned (NaN bf16 and fp32 values, out-of-range parents and tokens),
    so a kernel that reads padding fails visibly."""
    ss = np.random.SeedSequence(seed)
    r_tree, r_len, r_page, r_q, r_kv, r_tree_kv, r_tok, r_logit, r_boost = [
        np.random.default_rng(s) for s in ss.spawn(9)]

    trees = [np.asarray(parent_fn(r_tree), dtype=np.int32) for _ in range(B)]
    assert all(1 <= len(t) <= N or (len(t) == 0) for t in trees)
    counts = np.array([len(t) for t in trees], dtype=np.int32)
    ragged = bool(B) and bool((counts < N).any())
    parent = np.full((B, N), -1, dtype=np.int32)
    for b, t in enumerate(trees):
        parent[b, :len(t)] = t

    if isinstance(kv_len, (int, np.integer)):
        lens = np.full(B, int(kv_len), dtype=np.int32)
    elif isinstance(kv_len, tuple):
        lo, hi = kv_len
        lens = r_len.integers(lo, hi + 1, size=B).astype(np.int32)
    else:
        lens = np.asarray(kv_len, dtype=np.int32)
    assert lens.shape == (B,)

    page_table, num_pages = paged_layout(r_page, lens, N, P)
    q = _normal_bf16(r_q, (B, N, Hq, D))
    k_cache = _normal_bf16(r_kv, (num_pages, P, Hkv, D))
    v_cache = _normal_bf16(r_kv, (num_pages, P, Hkv, D))
    k_tree = _normal_bf16(r_tree_kv, (B, N, Hkv, D))
    v_tree = _normal_bf16(r_tree_kv, (B, N, Hkv, D))
    if poison:
        poison_cache_tails(k_cache, v_cache, page_table, lens, P)

    draft = np.zeros((B, N), dtype=np.int32)
    for b in range(B):
        n = counts[b]
        draft[b, :n] = draft_tokens(r_tok, parent[b, :n], V, distinct_siblings)

    logits = None
    if with_logits:
        logits = r_logit.standard_normal(size=(B, N, V), dtype=np.float32)
        for b in range(B):
            n = counts[b]
            if boost_prob > 0.0:
                boost_logits(r_boost, logits[b, :n], parent[b, :n], draft[b, :n], boost_prob,
                             boost_amount)
            if forced_path is not None:
                for c in forced_path(parent[b, :n]):
                    logits[b, parent[b, c], draft[b, c]] += np.float32(1e9)

    if ragged:
        for b in range(B):
            n = counts[b]
            pad = np.arange(n, N)
            q[b, n:] = BF16_NAN
            k_tree[b, n:] = BF16_NAN
            v_tree[b, n:] = BF16_NAN
            parent[b, n:] = np.where(pad % 2 == 0, pad + 3, -7)    # outside [-1, i-1]
            draft[b, n:] = V + 11
            if logits is not None:
                logits[b, n:] = np.float32(np.nan)

    meta = {"seed": seed, "boost_prob": boost_prob, "boost_amount": boost_amount,
            "max_depth": [int(tree_depths(parent[b, :counts[b]]).max()) if counts[b] else -1
                          for b in range(B)]}
    return Workload(name, B, N, Hq, Hkv, D, P, V, q, k_tree, v_tree, k_cache, v_cache,
                    page_table, lens, parent, draft, logits, meta,
                    counts if ragged else None)


# --------------------------------------------------------------------------
# the five named presets
# --------------------------------------------------------------------------

PRESETS = ("tiny", "llama8b_bs1", "llama8b_bs16", "llama70b_bs8", "long_wide_bs4")
# Ragged forests of a fused verification (this round's tree plus the previous
# round's re-sampled tree per sequence, padded to N).
RAGGED_PRESETS = ("llama8b_bs16_fused",)
# The paper's own verification shape (§7.1: LLaMA-2-7B, multi-head attention,
# depth-3 trees at most 4 wide, 12 tokens verified per request, batches 2-16).
PAPER_PRESETS = ("llama2_7b_bs2", "llama2_7b_bs16")


def preset(name: str, *, poison: bool = False, with_logits: bool = True,
           B: int | None = None, boost_amount: float = 3.0,
           boost_prob: float | None = None) -> Workload:
    """The five Llama-shaped verification workloads. Preset k (1-based) uses
    seed k-1. `B` overrides the batch (a bounded sample of the same recipe);
    `boost_amount` and `boost_prob` override the draft-token boost (tests use
    +20 with probability 1 to force deep accepted paths)."""
    def bp(default):
        return default if boost_prob is None else boost_prob
    if name == "tiny":
        return make_workload(name, 0, B=B or 1, N=16, Hq=8, Hkv=8, D=64, kv_len=128,
                             parent_fn=lambda r: tree_uniform_forest(r, 16), V=1000,
                             boost_prob=0.0, distinct_siblings=False, poison=poison,
                             with_logits=with_logits)
    if name == "llama8b_bs1":
        return make_workload(name, 1, B=B or 1, N=64, Hq=32, Hkv=8, D=128, kv_len=2048,
                             parent_fn=lambda r: tree_topk_expansion(r, (4, 4, 2, 2, 1, 1), 64),
                             V=128256, boost_prob=bp(0.6), boost_amount=boost_amount,
                             poison=poison, with_logits=with_logits)
    if name == "llama8b_bs16":
        return make_workload(name, 2, B=B or 16, N=64, Hq=32, Hkv=8, D=128,
                             kv_len=(1024, 4096),
                             parent_fn=lambda r: tree_random_depth_capped(r, 64, 8),
                             V=128256, boost_prob=bp(0.6), boost_amount=boost_amount,
                             poison=poison, with_logits=with_logits)
    if name == "llama70b_bs8":
        return make_workload(name, 3, B=B or 8, N=128, Hq=64, Hkv=8, D=128, kv_len=8192,
                             parent_fn=lambda r: tree_random_depth_capped(r, 128, 10),
                             V=128256, boost_prob=bp(0.5), boost_amount=boost_amount,
                             poison=poison, with_logits=with_logits)
    if name == "llama8b_bs16_fused":
        return make_workload(name, 5, B=B or 16, N=64, Hq=32, Hkv=8, D=128,
                             kv_len=(1024, 4096),
                             parent_fn=lambda r: fusion_forest(r, (24, 48), (0, 16), 8),
                             V=128256, boost_prob=bp(0.6), boost_amount=boost_amount,
                             poison=poison, with_logits=with_logits)
    if name in ("llama2_7b_bs2", "llama2_7b_bs16"):
        return make_workload(name, 6 if name.endswith("bs2") else 7,
                             B=B or (2 if name.endswith("bs2") else 16), N=12, Hq=32, Hkv=32,
                             D=128, kv_len=(256, 2048),
                             parent_fn=lambda r: tree_frontier_expansion(r, 4, 3, 12),
                             V=32000, boost_prob=bp(0.6), boost_amount=boost_amount,
                             poison=poison, with_logits=with_logits)
    if name == "long_wide_bs4":
        return make_workload(name, 4, B=B or 4, N=256, Hq=32, Hkv=8, D=128, kv_len=32768,
                             parent_fn=lambda r: tree_random_depth_capped(r, 256, 12,
                                                                          root_children=8),
                             V=128256, boost_prob=bp(0.4), boost_amount=boost_amount,
                             poison=poison, with_logits=with_logits)
    raise KeyError(name)


PRESET_DOC = {
    "tiny": "batch 1, 8/8 heads, head_dim 64, prefix 128, 16-node forest "
            "(parent uniform in [-1, i-1]), vocab 1000, seed 0",
    "llama8b_bs1": "batch 1, 32/8 heads, head_dim 128, prefix 2048 in 16-token pages, "
                   "64-node top-k tree (4,4,2,2,1,1), vocab 128256, +3 boost w.p. 0.6",
    "llama8b_bs16": "batch 16, 32/8 heads, head_dim 128, prefix U[1024,4096], 64-node "
                    "random trees (depth <= 8), vocab 128256, +3 boost w.p. 0.6",
    "llama70b_bs8": "batch 8, 64/8 heads, head_dim 128, prefix 8192, 128-node random trees "
                    "(depth <= 10), vocab 128256, +3 boost w.p. 0.5",
    "long_wide_bs4": "batch 4, 32/8 heads, head_dim 128, prefix 32768, 256-node trees "
                     "(8 root children, depth <= 12), vocab 128256, +3 boost w.p. 0.4",
    "llama2_7b_bs2": "batch 2, 32/32 heads (MHA), head_dim 128, prefix U[256,2048], 12-node "
                     "trees of depth 3 at most 4 wide, vocab 32000, +3 boost w.p. 0.6, seed 6",
    "llama2_7b_bs16": "batch 16, 32/32 heads (MHA), head_dim 128, prefix U[256,2048], 12-node "
                      "trees of depth 3 at most 4 wide, vocab 32000, +3 boost w.p. 0.6, seed 7",
    "llama8b_bs16_fused": "batch 16, 32/8 heads, head_dim 128, prefix U[1024,4096], per "
                          "sequence a 24-48-node tree plus a 0-16-node re-sampled tree "
                          "(second root), padded to 64, vocab 128256, seed 5",
}


# ---------------------------------------------------------------------------
# Inputs of the draft-tree builder (token-info sampling, Alg. 1 of §5.2, with
# the hot-token table of §6.1): per-step draft logits, a root token per
# sequence, the hot-token list and the bf16 token-info table over it.
@dataclass
class TreeBuildInputs:
    name: str
    B: int
    S: int          # speculative steps (rows of draft logits per sequence)
    V: int
    H: int          # hot tokens (0: no token information)
    k: int          # branch number
    budget: int     # verification token budget
    logits: np.ndarray     # [B, S, V] float32
    root: np.ndarray       # [B] int32
    table: np.ndarray      # [H, H] uint16 (bf16 bits)
    hot_vocab: np.ndarray  # [H] int32, distinct vocabulary ids
    hot_index: np.ndarray  # [V] int32, -1 for tokens without token-info


def make_tree_build_inputs(name: str, seed: int, *, B: int, S: int, V: int, H: int, k: int,
                           budget: int, logit_scale: float = 2.5,
                           info_scale: float = 1.0) -> TreeBuildInputs:
    """Seeded synthetic builder inputs. Draft logits are N(0, logit_scale^2)
    (peaked enough that a few tokens carry most of the mass); the hot set is a
    seeded random subset of the vocabulary (a stand-in for the corpus
    frequency ranking of §6.1); table entries are uniform with standard
    deviation info_scale, cut to bf16; roots are hot tokens with probability
    0.75."""
    ss = np.random.SeedSequence(seed)
    r_log, r_hot, r_tab, r_root = (np.random.default_rng(s) for s in ss.spawn(4))
    logits = np.empty((B, S, V), dtype=np.float32)
    for b in range(B):
        logits[b] = r_log.standard_normal((S, V), dtype=np.float32) * np.float32(logit_scale)
    hot_vocab = r_hot.permutation(V)[:H].astype(np.int32)
    hot_index = np.full(V, -1, dtype=np.int32)
    hot_index[hot_vocab] = np.arange(H, dtype=np.int32)
    table = np.empty((H, H), dtype=np.uint16)
    step = max(1, (1 << 24) // max(H, 1))
    for r0 in range(0, H, step):
        r1 = min(H, r0 + step)
        x = r_tab.random((r1 - r0, H), dtype=np.float32)
        x = (x - np.float32(0.5)) * np.float32(2.0 * 3.0 ** 0.5 * info_scale)
        table[r0:r1] = (x.view(np.uint32) >> 16).astype(np.uint16)     # bf16 by truncation
    root = r_root.integers(0, V, B).astype(np.int32)
    if H > 0:
        use_hot = r_root.random(B) < 0.75
        root[use_hot] = hot_vocab[r_root.integers(0, H, int(use_hot.sum()))]
    return TreeBuildInputs(name, B, S, V, H, k, budget, logits, root, table, hot_vocab,
                           hot_index)


TREE_BUILD_PRESETS = {
    # name: (seed, B, S, V, H, k, budget); "rs_" presets re-sample (Alg. 2)
    "tb_tiny": (40, 2, 3, 300, 60, 3, 16),
    "rs_llama8b_bs16": (43, 16, 7, 128256, 32768, 8, 64),
    "tb_llama2_bs16": (41, 16, 7, 32000, 32000, 8, 64),
    "tb_llama8b_bs16": (42, 16, 7, 128256, 32768, 8, 64),
}

TREE_BUILD_DOC = {
    "tb_tiny": "batch 2, 3 steps, vocab 300 with 60 hot tokens, k 3, budget 16",
    "tb_llama2_bs16": "batch 16, 7 steps, vocab 32000 (all hot: below the 40K threshold of "
                      "§6.1), k 8, budget 64",
    "tb_llama8b_bs16": "batch 16, 7 steps, vocab 128256 with the 32768 hot tokens of §6.1, "
                       "k 8, budget 64",
    "rs_llama8b_bs16": "re-sampling after verification at the tb_llama8b_bs16 shapes: accept "
                       "lengths U{1..4} (seeded), bonus tokens hot w.p. 0.75, threshold r = 1",
}


def resample_inputs(x: TreeBuildInputs, seed: int):
    """Verification outcome that drives re-sampling: accept lengths U{1..4}
    (the root plus up to three accepted drafts) and bonus tokens, hot with
    probability 0.75."""
    rng = np.random.default_rng(seed)
    alen = rng.integers(1, 5, x.B).astype(np.int32)
    bonus = rng.integers(0, x.V, x.B).astype(np.int32)
    if x.H > 0:
        hot = rng.random(x.B) < 0.75
        bonus[hot] = x.hot_vocab[rng.integers(0, x.H, int(hot.sum()))]
    return bonus, alen


def tree_build_preset(name: str) -> TreeBuildInputs:
    seed, B, S, V, H, k, budget = TREE_BUILD_PRESETS[name]
    return make_tree_build_inputs(name, seed, B=B, S=S, V=V, H=H, k=k, budget=budget)


# ---------------------------------------------------------------------------
# Inputs of the LM head fused with greedy verification: every tree node's final
# hidden state and the target model's LM-head weight, plus the draft trees.
@dataclass
class LmHeadInputs:
    name: str
    B: int
    N: int
    V: int
    d: int
    hidden: np.ndarray     # [B, N, d] uint16 (bf16 bits)
    w_head: np.ndarray     # [V, d] uint16 (bf16 bits), row v = token v
    parent: np.ndarray     # [B, N] int32
    draft: np.ndarray      # [B, N] int32
    num_nodes: np.ndarray | None   # [B] int32, or None (N nodes each)
    planted: np.ndarray    # [B, N] int32: token whose logit was raised, -1 if none


def _uniform_bf16(rng: np.random.Generator, shape, std: float, rows_per_chunk: int = 8192):
    """Uniform(-sqrt(3) std, sqrt(3) std) cut to bf16 by truncation, drawn in
    row chunks (the full 8B-shaped head is 128256 x 4096)."""
    out = np.empty(shape, dtype=np.uint16)
    a = np.float32(2.0 * 3.0 ** 0.5 * std)
    for r0 in range(0, shape[0], rows_per_chunk):
        r1 = min(shape[0], r0 + rows_per_chunk)
        x = (rng.random((r1 - r0,) + tuple(shape[1:]), dtype=np.float32) - np.float32(0.5)) * a
        out[r0:r1] = (x.view(np.uint32) >> 16).astype(np.uint16)
    return out


def make_lm_head_inputs(name: str, seed: int, *, B: int, N: int, V: int, d: int,
                        w_std: float = 0.02, plant_prob: float = 0.6, plant_gain: float = 6.0,
                        depth_lt: int = 8, num_nodes=None) -> LmHeadInputs:
    """Seeded synthetic inputs. Hidden states are N(0, 1) (a normalised final
    hidden state), the head is uniform with standard deviation w_std, so the
    logits spread with standard deviation about sqrt(d) w_std. Trees are
    depth-capped random trees (as in the llama8b_bs16 verification preset);
    for each node with children, with probability plant_prob the hidden state
    is moved along the head row of one random child's draft token so that this
    token's logit rises by about plant_gain (the child becomes acceptable, as
    a good draft would be). `num_nodes` (optional [B]) makes the batch ragged;
    padding rows keep random data."""
    ss = np.random.SeedSequence(seed)
    r_tree, r_tok, r_h, r_w, r_plant = (np.random.default_rng(s) for s in ss.spawn(5))
    counts = (np.full(B, N, dtype=np.int32) if num_nodes is None
              else np.asarray(num_nodes, dtype=np.int32))
    parent = np.full((B, N), -1, dtype=np.int32)
    draft = np.zeros((B, N), dtype=np.int32)
    for b in range(B):
        n = int(counts[b])
        if n:
            parent[b, :n] = tree_random_depth_capped(r_tree, n, depth_lt)
            draft[b, :n] = draft_tokens(r_tok, parent[b, :n], V, True)
    w_bits = _uniform_bf16(r_w, (V, d), w_std)
    h = r_h.standard_normal((B, N, d), dtype=np.float32)
    planted = np.full((B, N), -1, dtype=np.int32)
    for b in range(B):
        n = int(counts[b])
        kids: dict[int, list] = {}
        for i in range(n):
            if parent[b, i] >= 0:
                kids.setdefault(int(parent[b, i]), []).append(i)
        for p in range(n):
            ch = kids.get(p)
            if ch and r_plant.random() < plant_prob:
                t = int(draft[b, ch[int(r_plant.integers(0, len(ch)))]])
                wt = bf16_bits_to_f32(w_bits[t]).astype(np.float64)
                h[b, p] += np.float32(plant_gain / max(float(wt @ wt), 1e-30)) * wt.astype(np.float32)
                planted[b, p] = t
    return LmHeadInputs(name, B, N, V, d, f32_to_bf16_bits(h), w_bits, parent, draft,
                        None if num_nodes is None else counts, planted)


LM_HEAD_PRESETS = {
    # name: (seed, B, N, V, d)
    "lm_tiny": (50, 2, 16, 1000, 256),
    "lm_llama8b_bs16": (51, 16, 64, 128256, 4096),
}

LM_HEAD_DOC = {
    "lm_tiny": "batch 2, 16-node trees, vocab 1000, hidden size 256",
    "lm_llama8b_bs16": "batch 16, 64-node random trees (depth <= 8), vocab 128256, hidden "
                       "size 4096 (Llama-3-8B's LM head), planted acceptable drafts w.p. 0.6",
}


def lm_head_preset(name: str) -> LmHeadInputs:
    seed, B, N, V, d = LM_HEAD_PRESETS[name]
    return make_lm_head_inputs(name, seed, B=B, N=N, V=V, d=d)
