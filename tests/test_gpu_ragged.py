"""GPU parity for ragged batches (verification fusion, §6.2): each sequence
carries a forest of its own size, padded to N with poisoned inputs (NaN
values, out-of-range parents and tokens). Compared with the oracle given the
same node counts; padding rows must come out exactly as zeros / lse -inf /
argmax -1, and nothing of the padding may leak into a real row."""
import numpy as np
import pytest
import torch

from paper_2602_21224_amd import workloads as W
from tests import gpu_util as U

pytestmark = pytest.mark.gpu


def forest_wl(seed, *, B, N, Hq, Hkv, D, L, P=16, primary=(1, 30), resampled=(0, 12),
              empty=0.15, with_logits=False, V=64, depth=6):
    def fn(r):
        if r.random() < empty:
            return np.zeros(0, dtype=np.int32)
        t = W.fusion_forest(r, primary, resampled, depth)
        return t[:N]
    return W.make_workload("forest", seed, B=B, N=N, Hq=Hq, Hkv=Hkv, D=D, kv_len=L,
                           parent_fn=fn, V=V, P=P, poison=True, with_logits=with_logits,
                           boost_prob=0.8, boost_amount=6.0)


def attention_compare(oracle_mod, T, w, label):
    print(f"case {label}: B={w.B} N={w.N} Hq={w.Hq} Hkv={w.Hkv} D={w.D} P={w.P} "
          f"nodes={w.num_nodes.tolist()[:8]}", flush=True)
    got, glse = U.gpu_attention(T, w)
    nn = w.num_nodes
    for b in range(w.B):
        n = int(nn[b])
        assert (got[b, n:] == 0).all() and np.isneginf(glse[b, n:]).all(), (label, b)
        assert np.isfinite(got[b, :n]).all() and np.isfinite(glse[b, :n]).all(), (label, b)
    want, wlse = oracle_mod.tree_attention(w.q, w.k_tree, w.v_tree, w.k_cache, w.v_cache,
                                           w.page_table, w.kv_len, w.parent, num_nodes=nn)
    mask = np.arange(w.N)[None, :] < nn[:, None]              # real nodes
    U.assert_attention_close(got[mask], want[mask], glse[mask], wlse[mask], label)


CASES = [
    # (B, N, Hq, Hkv, D, L, P)
    (5, 24, 8, 2, 64, (0, 150), 16),
    (4, 40, 32, 8, 128, (40, 400), 16),
    (3, 64, 32, 8, 128, (500, 1500), 16),
    (6, 30, 16, 4, 128, (0, 90), 1),          # pages shorter than a load block
    (2, 256, 64, 8, 128, (100, 300), 16),     # several row blocks; their count varies per sequence
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_ragged_attention(oracle_mod, case):
    T = U.require_gpu()
    B, N, Hq, Hkv, D, L, P = CASES[case]
    primary = (1, min(N, 200))
    w = forest_wl(300 + case, B=B, N=N, Hq=Hq, Hkv=Hkv, D=D, L=L, P=P, primary=primary,
                  resampled=(0, max(1, N // 4)))
    assert w.num_nodes is not None
    attention_compare(oracle_mod, T, w, f"ragged{case}")


def test_all_sequences_empty(oracle_mod):
    T = U.require_gpu()
    w = forest_wl(330, B=3, N=16, Hq=8, Hkv=8, D=64, L=(10, 80), empty=1.0)
    assert (w.num_nodes == 0).all()
    got, glse = U.gpu_attention(T, w)
    assert (got == 0).all() and np.isneginf(glse).all()


def test_fused_preset_all_outputs(oracle_mod):
    T = U.require_gpu()
    w = W.preset("llama8b_bs16_fused", poison=True, with_logits=False)
    attention_compare(oracle_mod, T, w, "llama8b_bs16_fused")


def test_ragged_matches_dense_on_each_sequence():
    """A ragged call gives, for every sequence's real nodes, exactly the result
    of a dense call on that sequence alone (same kernels, bit for bit is not
    required: the split of keys over workgroups differs)."""
    T = U.require_gpu()
    w = forest_wl(340, B=4, N=48, Hq=32, Hkv=8, D=128, L=(200, 900), empty=0.0)
    got, glse = U.gpu_attention(T, w)
    for b in range(w.B):
        n = int(w.num_nodes[b])
        w1 = W.Workload("one", 1, n, w.Hq, w.Hkv, w.D, w.P, w.V, w.q[b:b + 1, :n].copy(),
                        w.k_tree[b:b + 1, :n].copy(), w.v_tree[b:b + 1, :n].copy(), w.k_cache,
                        w.v_cache, w.page_table[b:b + 1].copy(), w.kv_len[b:b + 1].copy(),
                        w.parent[b:b + 1, :n].copy(), w.draft[b:b + 1, :n].copy(), None)
        g1, l1 = U.gpu_attention(T, w1)
        U.assert_attention_close(got[b:b + 1, :n], g1, glse[b:b + 1, :n], l1, f"alone{b}")


def test_ragged_argmax_accept_and_compaction(oracle_mod):
    T = U.require_gpu()
    w = forest_wl(350, B=9, N=40, Hq=8, Hkv=4, D=64, L=(0, 60), with_logits=True, V=3000,
                  primary=(1, 28), resampled=(0, 12))
    d = U.upload(w)
    amax, alen, aidx, bonus = T.tree_argmax_accept(U.dev(w.logits), U.dev(w.draft), d["parent"],
                                                   num_nodes=d["num_nodes"])
    torch.cuda.synchronize()
    amax, alen, aidx, bonus = (t.cpu().numpy() for t in (amax, alen, aidx, bonus))
    want_am = oracle_mod.argmax(np.nan_to_num(w.logits, nan=0.0))
    for b in range(w.B):
        n = int(w.num_nodes[b])
        assert np.array_equal(amax[b, :n], want_am[b, :n]) and (amax[b, n:] == -1).all()
    wl, wi, wb = oracle_mod.accept(w.draft, w.parent, amax, num_nodes=w.num_nodes)
    assert np.array_equal(alen, wl) and np.array_equal(aidx, wi) and np.array_equal(bonus, wb)
    assert (alen[w.num_nodes == 0] == 0).all() and (bonus[w.num_nodes == 0] == -1).all()
    kc, vc = d["k_cache"].clone(), d["v_cache"].clone()
    T.kv_compact_accepted(d["k_tree"], d["v_tree"], kc, vc, d["page_table"], d["kv_len"],
                          U.dev(aidx), U.dev(alen))
    torch.cuda.synchronize()
    wk, wv = oracle_mod.kv_compact(w.k_tree, w.v_tree, w.k_cache, w.v_cache, w.page_table,
                                   w.kv_len, aidx, alen)
    assert np.array_equal(kc.view(torch.int16).cpu().numpy().view(np.uint16), wk)
    assert np.array_equal(vc.view(torch.int16).cpu().numpy().view(np.uint16), wv)


def test_validate_ragged():
    """The contract check skips padding (whose parents are poisoned) only when
    it is given the node counts, and flags counts outside [0, N]."""
    T = U.require_gpu()
    w = forest_wl(41, B=6, N=40, Hq=8, Hkv=2, D=64, L=np.array([0, 17, 64, 5, 300, 33]))
    print(f"case validate: nodes={w.num_nodes.tolist()}", flush=True)
    pt, kl, par = U.dev(w.page_table), U.dev(w.kv_len), U.dev(w.parent)
    ok = T.tv_validate_inputs(pt, kl, par, P=w.P, num_pages=w.num_pages,
                              num_nodes=U.dev(w.num_nodes))
    assert int(ok.item()) == 0
    assert (w.num_nodes < w.N).any() and w.num_nodes.max() >= 1
    dense = T.tv_validate_inputs(pt, kl, par, P=w.P, num_pages=w.num_pages)
    assert int(dense.item()) & 1                   # padding parents point forward
    bad_nn = w.num_nodes.copy(); bad_nn[2] = w.N + 1
    st = T.tv_validate_inputs(pt, kl, par, P=w.P, num_pages=w.num_pages, num_nodes=U.dev(bad_nn))
    assert int(st.item()) == 16
    b = int(np.argmax(w.num_nodes))
    bad_par = w.parent.copy(); bad_par[b, w.num_nodes[b] - 1] = w.num_nodes[b] + 2
    st = T.tv_validate_inputs(pt, kl, U.dev(bad_par), P=w.P, num_pages=w.num_pages,
                              num_nodes=U.dev(w.num_nodes))
    assert int(st.item()) == 1
