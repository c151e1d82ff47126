"""GPU parity of tree_argmax_accept and kv_compact_accepted against the CPU
oracle (through the C ABI). Both must match bit for bit."""
import numpy as np
import pytest
import torch

from paper_2602_21224_amd import workloads as W
from tests import gpu_util as U

pytestmark = pytest.mark.gpu


def gpu_accept(T, logits, draft, parent):
    a, alen, aidx, bonus = T.tree_argmax_accept(U.dev(logits), U.dev(draft), U.dev(parent))
    torch.cuda.synchronize()
    return a.cpu().numpy(), alen.cpu().numpy(), aidx.cpu().numpy(), bonus.cpu().numpy()


def check_accept(oracle_mod, T, logits, draft, parent, label):
    print(f"case {label}: B={parent.shape[0]} N={parent.shape[1]} V={logits.shape[-1]}",
          flush=True)
    a, alen, aidx, bonus = gpu_accept(T, logits, draft, parent)
    ra = oracle_mod.argmax(logits)
    np.testing.assert_array_equal(a, ra)
    rl, ri, rb = oracle_mod.accept(draft, parent, ra)
    np.testing.assert_array_equal(alen, rl)
    np.testing.assert_array_equal(aidx, ri)
    np.testing.assert_array_equal(bonus, rb)
    hist = np.bincount(alen)
    print(f"[{label}] accept_len histogram {hist.tolist()}", flush=True)
    return a, alen, aidx


@pytest.mark.parametrize("name", W.PRESETS + W.PAPER_PRESETS)
def test_presets(oracle_mod, name):
    T = U.require_gpu()
    w = W.preset(name)
    check_accept(oracle_mod, T, w.logits, w.draft, w.parent, name)


def test_forced_deep_paths(oracle_mod):
    """+20 boosts on every node make long accepted paths and many ties among
    matching siblings' subtrees."""
    T = U.require_gpu()
    w = W.preset("llama8b_bs16", boost_amount=20.0)
    w2 = W.make_workload("forced", 9, B=8, N=64, Hq=1, Hkv=1, D=64, kv_len=10,
                         parent_fn=lambda r: W.tree_random_depth_capped(r, 64, 8), V=5000,
                         boost_prob=1.0, boost_amount=20.0)
    check_accept(oracle_mod, T, w.logits, w.draft, w.parent, "boost20")
    _, alen2, _ = check_accept(oracle_mod, T, w2.logits, w2.draft, w2.parent, "boost20-small")
    assert alen2.max() >= 4


def test_chain_star_single_and_ragged_vocab(oracle_mod):
    T = U.require_gpu()
    rng = np.random.default_rng(5)
    for N, parent_row, V in ((256, W.tree_chain(256), 7), (33, W.tree_star(33), 130),
                             (1, np.array([-1], np.int32), 1), (50, W.tree_chain(50), 129001)):
        B = 3
        parent = np.stack([parent_row] * B)
        draft = rng.integers(0, min(V, 3), size=(B, N)).astype(np.int32)
        logits = rng.standard_normal((B, N, V), dtype=np.float32)
        # make the chain's argmax follow the draft for a while
        for b in range(B):
            for i in range(min(N - 1, 5 * (b + 1))):
                logits[b, i, draft[b, i + 1]] += 50.0
        check_accept(oracle_mod, T, logits, draft, parent, f"N{N}V{V}")


def test_ties_signed_zero_and_nan(oracle_mod):
    T = U.require_gpu()
    V = 10000
    logits = np.zeros((1, 6, V), np.float32) - 5.0
    logits[0, 0, [17, 4000, 9999]] = 2.0            # tie -> 17
    logits[0, 1, :] = -0.0
    logits[0, 1, 5000] = 0.0                        # -0 == +0 -> index 0
    logits[0, 2, [3, 7000]] = np.nan                # first NaN -> 3
    logits[0, 2, 10] = np.inf
    logits[0, 3, :] = -np.inf                       # all -inf -> 0
    logits[0, 4, 4096] = np.inf                     # segment boundary region
    logits[0, 4, 4095] = np.inf
    logits[0, 5, V - 1] = 1.0
    parent = np.array([[-1, 0, 1, 2, 3, 4]], np.int32)
    draft = np.array([[0, 17, 0, 3, 0, 4095]], np.int32)
    check_accept(oracle_mod, T, logits, draft, parent, "special")


def test_unaligned_vocab_rows(oracle_mod):
    T = U.require_gpu()
    rng = np.random.default_rng(9)
    for V in (1, 2, 3, 5, 4097, 32003):
        logits = rng.standard_normal((2, 7, V), dtype=np.float32)
        parent = np.stack([W.tree_uniform_forest(rng, 7) for _ in range(2)])
        draft = rng.integers(0, V, size=(2, 7)).astype(np.int32)
        check_accept(oracle_mod, T, logits, draft, parent, f"V{V}")


def _compact_case(oracle_mod, T, w, alen, aidx, label):
    print(f"case {label}: compaction, accept_len {alen.tolist()[:16]}", flush=True)
    kc, vc = U.dev_bf16(w.k_cache), U.dev_bf16(w.v_cache)
    T.kv_compact_accepted(U.dev_bf16(w.k_tree), U.dev_bf16(w.v_tree), kc, vc,
                          U.dev(w.page_table), U.dev(w.kv_len), U.dev(aidx), U.dev(alen))
    torch.cuda.synchronize()
    got_k = kc.view(torch.int16).cpu().numpy().view(np.uint16)
    got_v = vc.view(torch.int16).cpu().numpy().view(np.uint16)
    rk, rv = oracle_mod.kv_compact(w.k_tree, w.v_tree, w.k_cache, w.v_cache, w.page_table,
                                   w.kv_len, aidx, alen)
    assert np.array_equal(got_k, rk) and np.array_equal(got_v, rv)


@pytest.mark.parametrize("name", W.PRESETS + W.PAPER_PRESETS)
def test_accept_then_compaction_forced_paths(oracle_mod, name):
    """Every preset with a +20 boost on one child of every internal node, so
    accepted paths run down to the trees' depth caps: the GPU's argmax/accept
    must equal the oracle's, and the GPU's compaction of the GPU's accepted
    paths must equal the oracle's compaction byte for byte."""
    T = U.require_gpu()
    w = W.preset(name, poison=True, boost_amount=20.0, boost_prob=1.0)
    _, alen, aidx = check_accept(oracle_mod, T, w.logits, w.draft, w.parent, f"{name}+20")
    if name != "tiny":
        deep = min(5, max(w.meta["max_depth"]) + 1)
        assert alen.max() >= deep, f"{name}: the forced boosts should give deep paths"
    _compact_case(oracle_mod, T, w, alen, aidx, name)


def test_compaction_crosses_pages_and_len_one(oracle_mod):
    T = U.require_gpu()
    w = W.make_workload("c", 77, B=5, N=40, Hq=8, Hkv=8, D=128, kv_len=[0, 15, 16, 17, 31],
                        parent_fn=lambda r: W.tree_chain(40), V=50, P=16, poison=True)
    alen = np.array([40, 1, 17, 2, 33], np.int32)
    aidx = np.full((5, 40), -1, np.int32)
    for b in range(5):
        aidx[b, :alen[b]] = np.arange(alen[b])
    _compact_case(oracle_mod, T, w, alen, aidx, "pages")


def test_validate_inputs():
    T = U.require_gpu()
    w = W.preset("llama8b_bs16", with_logits=False, B=4)
    ok = T.tv_validate_inputs(U.dev(w.page_table), U.dev(w.kv_len), U.dev(w.parent), P=w.P,
                              num_pages=w.num_pages)
    assert int(ok.item()) == 0
    bad_parent = w.parent.copy(); bad_parent[1, 5] = 7
    bad_pt = w.page_table.copy(); bad_pt[2, 0] = w.num_pages
    st = T.tv_validate_inputs(U.dev(bad_pt), U.dev(w.kv_len), U.dev(bad_parent), P=w.P,
                              num_pages=w.num_pages)
    assert int(st.item()) == (1 | 8)


def test_unrelated_runtime_error_is_not_reported(oracle_mod):
    """An error left in the HIP runtime by an earlier, unrelated call of the
    caller's neither turns correct calls into failures nor is consumed by them:
    every launch is checked by its own status."""
    import ctypes
    T = U.require_gpu()
    hip = None
    with open("/proc/self/maps") as fh:
        for line in fh:
            if "libamdhip64" in line:
                hip = ctypes.CDLL(line.split()[-1])
                break
    assert hip is not None
    w = W.preset("tiny")
    d = U.upload(w)
    logits, draft, parent = U.dev(w.logits), U.dev(w.draft), U.dev(w.parent)
    out = torch.empty((w.B, w.N, w.Hq, w.D), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((w.B, w.N, w.Hq), dtype=torch.float32, device="cuda")
    amax = torch.empty((w.B, w.N), dtype=torch.int32, device="cuda")
    alen = torch.empty((w.B,), dtype=torch.int32, device="cuda")
    aidx = torch.empty((w.B, w.N), dtype=torch.int32, device="cuda")
    bonus = torch.empty((w.B,), dtype=torch.int32, device="cuda")
    ws_a = torch.empty(T.attention_workspace_size(w.B, w.N, w.Hq, w.Hkv, w.D), dtype=torch.uint8,
                       device="cuda")
    ws_m = torch.empty(T.argmax_workspace_size(w.B, w.N, w.V), dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    print("case stale error: hipSetDevice(99999) before the calls", flush=True)
    assert hip.hipSetDevice(ctypes.c_int(99999)) != 0      # host-side check, nothing launched
    try:
        T.tree_argmax_accept(logits, draft, parent, argmax_out=amax, accept_len=alen,
                             accept_idx=aidx, bonus_token=bonus, workspace=ws_m)
        T.tree_verify_attention(d["q"], d["k_tree"], d["v_tree"], d["k_cache"], d["v_cache"],
                                d["page_table"], d["kv_len"], d["parent"], max_kv_len=w.max_kv_len,
                                out=out, lse=lse, workspace=ws_a)
        assert hip.hipPeekAtLastError() != 0               # still the caller's to collect
    finally:
        hip.hipGetLastError()
    torch.cuda.synchronize()
    ra = oracle_mod.argmax(w.logits)
    np.testing.assert_array_equal(amax.cpu().numpy(), ra)
    rl, ri, rb = oracle_mod.accept(w.draft, w.parent, ra)
    np.testing.assert_array_equal(alen.cpu().numpy(), rl)
    np.testing.assert_array_equal(aidx.cpu().numpy(), ri)
    np.testing.assert_array_equal(bonus.cpu().numpy(), rb)
    want, wlse = oracle_mod.tree_attention(w.q, w.k_tree, w.v_tree, w.k_cache, w.v_cache,
                                           w.page_table, w.kv_len, w.parent)
    U.assert_attention_close(U.bf16_to_f64(out), want, lse.cpu().numpy().astype(np.float64), wlse,
                             "stale-error")
