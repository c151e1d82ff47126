"""GPU parity of tree_verify_attention against the CPU oracle (through the C ABI).

Every output (out and lse) is compared element by element with the oracle,
on small shapes and on the five Llama-shaped workloads at full size, in the
launch configuration the benchmark times; properties that hold at any size
(determinism, page-permutation invariance, no leakage from invisible tree
rows) are checked on top.
"""
import numpy as np
import pytest
import torch

from paper_2602_21224_amd import workloads as W
from tests import gpu_util as U

pytestmark = pytest.mark.gpu


def wl(seed, *, B, N, Hq, Hkv, D, L, P=16, tree="forest", poison=True, depth=6, V=64):
    fns = {
        "forest": lambda r: W.tree_uniform_forest(r, N),
        "chain": lambda r: W.tree_chain(N),
        "star": lambda r: W.tree_star(N),
        "capped": lambda r: W.tree_random_depth_capped(r, N, depth),
    }
    return W.make_workload("t", seed, B=B, N=N, Hq=Hq, Hkv=Hkv, D=D, kv_len=L,
                           parent_fn=fns[tree], V=V, P=P, poison=poison, with_logits=False)


def full_compare(oracle_mod, T, w, label, scale=0.0):
    print(f"case {label}: B={w.B} N={w.N} Hq={w.Hq} Hkv={w.Hkv} D={w.D} P={w.P} "
          f"kv_len={w.kv_len.tolist()[:8]}", flush=True)
    got, glse = U.gpu_attention(T, w, scale=scale)
    want, wlse = oracle_mod.tree_attention(w.q, w.k_tree, w.v_tree, w.k_cache, w.v_cache,
                                           w.page_table, w.kv_len, w.parent, scale=scale,
                                           num_nodes=w.num_nodes)
    if w.num_nodes is not None:
        # padding rows are exact: zeros, lse -inf; compare the rest numerically
        for b in range(w.B):
            n = int(w.num_nodes[b])
            assert (got[b, n:] == 0).all() and np.isneginf(glse[b, n:]).all(), (label, b)
            glse[b, n:] = 0.0
            wlse[b, n:] = 0.0
    U.assert_attention_close(got, want, glse, wlse, label)


SMALL = [
    # (B, N, Hq, Hkv, D, L, P, tree)
    (1, 16, 8, 8, 64, 128, 16, "forest"),       # the tiny preset's shape
    (3, 7, 4, 4, 64, (0, 100), 16, "forest"),
    (2, 1, 8, 2, 128, (0, 70), 16, "forest"),   # single node = decode
    (2, 33, 8, 2, 128, (1, 97), 4, "capped"),
    (2, 64, 32, 8, 128, (31, 33), 16, "capped"),
    (2, 64, 32, 8, 128, (200, 700), 16, "capped"),
    (1, 100, 8, 1, 64, 300, 1, "forest"),       # G = 8, P = 1
    (2, 40, 12, 4, 128, (50, 90), 8, "star"),   # G = 3: rows of a node straddle waves
    (1, 256, 8, 8, 64, 64, 64, "chain"),        # deepest chain, large pages
    (1, 256, 16, 8, 128, 33, 16, "capped"),     # 512 rows: two row blocks
    (1, 128, 64, 8, 128, 0, 16, "capped"),      # empty prefix, 4 row blocks
    (4, 9, 4, 2, 64, (0, 3), 16, "forest"),     # prefixes shorter than a tile
    (2, 16, 8, 8, 128, (100, 900), 16, "capped"),   # 16 rows per KV head: the narrow-unit path
    (3, 5, 6, 2, 128, (0, 300), 2, "forest"),   # 15 narrow rows, G = 3, two-key pages
]


@pytest.mark.parametrize("case", range(len(SMALL)))
def test_small_shapes_all_outputs(oracle_mod, case):
    T = U.require_gpu()
    B, N, Hq, Hkv, D, L, P, tree = SMALL[case]
    w = wl(100 + case, B=B, N=N, Hq=Hq, Hkv=Hkv, D=D, L=L, P=P, tree=tree)
    full_compare(oracle_mod, T, w, f"small{case}")


def test_explicit_scale(oracle_mod):
    T = U.require_gpu()
    w = wl(7, B=2, N=20, Hq=8, Hkv=2, D=128, L=(40, 90), tree="capped")
    full_compare(oracle_mod, T, w, "scale0.05", scale=0.05)


def test_tiny_preset(oracle_mod):
    T = U.require_gpu()
    full_compare(oracle_mod, T, W.preset("tiny", poison=True, with_logits=False), "tiny")


def test_llama8b_bs1_preset_all_outputs(oracle_mod):
    T = U.require_gpu()
    full_compare(oracle_mod, T, W.preset("llama8b_bs1", poison=True, with_logits=False),
                 "llama8b_bs1")


@pytest.mark.parametrize("name", ["llama8b_bs16", "llama70b_bs8", "long_wide_bs4"])
def test_full_size_presets_all_outputs(oracle_mod, name):
    """Configs 3-5 at full size: every out and lse element against the oracle."""
    T = U.require_gpu()
    w = W.preset(name, poison=True, with_logits=False)
    full_compare(oracle_mod, T, w, name)


@pytest.mark.parametrize("name", W.PAPER_PRESETS)
def test_paper_shape_presets_all_outputs(oracle_mod, name):
    """The paper's own verification shape (multi-head attention, 12-node trees of
    depth 3 at most 4 wide): 12 query rows per KV head."""
    T = U.require_gpu()
    w = W.preset(name, poison=True, with_logits=False)
    full_compare(oracle_mod, T, w, name)


@pytest.mark.parametrize("B,N,Hq,Hkv,L,P", [
    (2, 12, 8, 2, (1500, 3000), 1),    # pages of one key: a 512-key page-id window
    (2, 9, 8, 2, (1600, 2900), 2),     # pages of two keys: 1024-key windows
    (1, 16, 16, 4, 9000, 16),          # 16-key pages: crosses the 8192-key window once
    (2, 12, 4, 4, (1500, 3000), 1),    # 12 rows per KV head (narrow units) over one-key pages
])
def test_page_id_windows(oracle_mod, B, N, Hq, Hkv, L, P):
    """Pieces whose prefix spans more page ids than the kernel caches at once run in
    several windows that carry the softmax state across; every output crosses at
    least one window boundary."""
    T = U.require_gpu()
    w = wl(71 + P, B=B, N=N, Hq=Hq, Hkv=Hkv, D=128, L=L, P=P, tree="capped")
    full_compare(oracle_mod, T, w, f"window_P{P}")


def test_page_permutation_and_determinism():
    """Physically permuting pages (and the table) changes nothing, bit for bit,
    and two runs are bit-identical."""
    T = U.require_gpu()
    w = W.preset("llama8b_bs16", poison=True, with_logits=False, B=4)
    a, la = U.gpu_attention(T, w)
    b, lb = U.gpu_attention(T, w)
    assert np.array_equal(a, b) and np.array_equal(la, lb)
    perm = np.random.default_rng(3).permutation(w.num_pages)
    kc = np.empty_like(w.k_cache); kc[perm] = w.k_cache
    vc = np.empty_like(w.v_cache); vc[perm] = w.v_cache
    pt = np.where(w.page_table >= 0, perm[np.maximum(w.page_table, 0)], -1).astype(np.int32)
    w.k_cache, w.v_cache, w.page_table = kc, vc, pt
    c, lc = U.gpu_attention(T, w)
    assert np.array_equal(a, c) and np.array_equal(la, lc)


def test_invisible_tree_rows_do_not_leak():
    """Poisoning every tree row that is not on node i's root path with +-1e4
    leaves node i's output unchanged (checked for the deepest node)."""
    T = U.require_gpu()
    from tests import bruteforce as BF
    w = wl(21, B=2, N=64, Hq=32, Hkv=8, D=128, L=(100, 300), tree="capped")
    a, _ = U.gpu_attention(T, w)
    for b in range(2):
        i = int(np.argmax(W.tree_depths(w.parent[b])))
        hide = ~BF.visibility_closure(w.parent[b])[i]
        kt, vt = w.k_tree.copy(), w.v_tree.copy()
        kt[b, hide] = W.f32_to_bf16_bits(np.float32(1e4))
        vt[b, hide] = W.f32_to_bf16_bits(np.float32(-1e4))
        w2 = wl(21, B=2, N=64, Hq=32, Hkv=8, D=128, L=(100, 300), tree="capped")
        w2.k_tree, w2.v_tree = kt, vt
        c, _ = U.gpu_attention(T, w2)
        assert np.array_equal(a[b, i], c[b, i])


def test_nondefault_stream(oracle_mod):
    T = U.require_gpu()
    w = wl(31, B=2, N=30, Hq=16, Hkv=4, D=128, L=(64, 200), tree="capped")
    d = U.upload(w)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        out, lse = T.tree_verify_attention(d["q"], d["k_tree"], d["v_tree"], d["k_cache"],
                                           d["v_cache"], d["page_table"], d["kv_len"],
                                           d["parent"], max_kv_len=w.max_kv_len)
    s.synchronize()
    want, wlse = oracle_mod.tree_attention(w.q, w.k_tree, w.v_tree, w.k_cache, w.v_cache,
                                           w.page_table, w.kv_len, w.parent)
    U.assert_attention_close(U.bf16_to_f64(out), want, lse.cpu().numpy(), wlse, "stream")


def test_understated_max_kv_len_hint_is_still_exact(oracle_mod):
    """The host-side length bound only sizes the launch; an understated bound
    must still give exact results."""
    T = U.require_gpu()
    w = wl(41, B=3, N=20, Hq=8, Hkv=2, D=128, L=(300, 900), tree="capped")
    d = U.upload(w)
    out, lse = T.tree_verify_attention(d["q"], d["k_tree"], d["v_tree"], d["k_cache"],
                                       d["v_cache"], d["page_table"], d["kv_len"], d["parent"],
                                       max_kv_len=0)
    want, wlse = oracle_mod.tree_attention(w.q, w.k_tree, w.v_tree, w.k_cache, w.v_cache,
                                           w.page_table, w.kv_len, w.parent)
    U.assert_attention_close(U.bf16_to_f64(out), want, lse.cpu().numpy(), wlse, "hint0")


def test_shared_workspace_alternating_inputs(oracle_mod):
    """One workspace reused by calls on different inputs of one shape (units
    split over several workgroups, so pieces meet in the workspace): every call
    matches the oracle on its own inputs, and repeats are bit-identical."""
    T = U.require_gpu()
    ws_ = [wl(51 + k, B=4, N=64, Hq=32, Hkv=8, D=128, L=(500, 2000), tree="capped") for k in range(2)]
    w0 = ws_[0]
    need = T.attention_workspace_size(w0.B, w0.N, w0.Hq, w0.Hkv, w0.D)
    work = torch.empty(need, dtype=torch.uint8, device="cuda")
    work.fill_(0xFF)                       # contents on entry must not matter
    dev_in = [U.upload(w) for w in ws_]
    want = [oracle_mod.tree_attention(w.q, w.k_tree, w.v_tree, w.k_cache, w.v_cache,
                                      w.page_table, w.kv_len, w.parent) for w in ws_]
    first = [None, None]
    for it in range(6):
        k = it % 2
        d, w = dev_in[k], ws_[k]
        out, lse = T.tree_verify_attention(d["q"], d["k_tree"], d["v_tree"], d["k_cache"],
                                           d["v_cache"], d["page_table"], d["kv_len"],
                                           d["parent"], max_kv_len=w.max_kv_len, workspace=work)
        torch.cuda.synchronize()
        got, glse = U.bf16_to_f64(out), lse.cpu().numpy().astype(np.float64)
        if first[k] is None:
            U.assert_attention_close(got, want[k][0], glse, want[k][1], f"alt{it}")
            first[k] = (got, glse)
        else:
            assert np.array_equal(got, first[k][0]) and np.array_equal(glse, first[k][1]), f"alt{it}"


@pytest.mark.parametrize("B,N,Hq,Hkv,D,L", [
    (130, 4, 8, 2, 64, (0, 200)),       # sequence count spans several 64-wide scan chunks
    (1024, 2, 4, 4, 64, (0, 70)),       # the largest supported batch
    (1, 256, 64, 8, 128, 300),          # (Hq / Hkv) * N = 2048 rows: eight row blocks
])
def test_batch_and_row_extremes(oracle_mod, B, N, Hq, Hkv, D, L):
    T = U.require_gpu()
    w = wl(61 + B, B=B, N=N, Hq=Hq, Hkv=Hkv, D=D, L=L, tree="capped")
    full_compare(oracle_mod, T, w, f"extreme_B{B}_N{N}_G{Hq // Hkv}")
