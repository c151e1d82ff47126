"""GPU parity of tree_build (token-info sampling, Alg. 1, with budget pruning,
§5.2) against the CPU oracle, through the C ABI.

Tokens, parents and node counts must match bit for bit: every decision is
either a ranking of fp32 logit sums (identical on both sides) or a ranking of
fp64 joint probabilities, and the oracle reports how far apart the competing
joints were; the cases below are asserted to have margins far above the
fp64 rounding of either side. Joint probabilities (fp32 output) match to
1e-6 relative."""
import numpy as np
import pytest
import torch

from paper_2602_21224_amd import workloads as W
from tests import gpu_util as U

pytestmark = pytest.mark.gpu


def run_gpu(T, x, budget=None, k=None):
    budget = x.budget if budget is None else budget
    k = x.k if k is None else k
    H = x.H
    tab = U.dev(x.table.view(np.int16)).view(torch.bfloat16) if H > 0 else None
    par, tok, jnt, nn = T.tree_build(U.dev(x.logits), U.dev(x.root), tab,
                                     U.dev(x.hot_vocab) if H > 0 else None,
                                     U.dev(x.hot_index) if H > 0 else None, k=k, budget=budget)
    torch.cuda.synchronize()
    return par.cpu().numpy(), tok.cpu().numpy(), jnt.cpu().numpy(), nn.cpu().numpy()


def compare(oracle_mod, T, x, label, budget=None, k=None):
    budget = x.budget if budget is None else budget
    k = x.k if k is None else k
    print(f"case {label}: B={x.B} S={x.S} V={x.V} H={x.H} k={k} budget={budget}", flush=True)
    margins = []
    want = oracle_mod.tree_build(x.logits, x.root, x.table, x.hot_vocab, k, budget, margins)
    if margins:
        assert min(margins) > 1e-9, f"{label}: near-tie in the oracle ({min(margins):.2e})"
    got = run_gpu(T, x, budget, k)
    np.testing.assert_array_equal(got[3], want[3], err_msg=f"{label} num_nodes")
    np.testing.assert_array_equal(got[1], want[1], err_msg=f"{label} token")
    np.testing.assert_array_equal(got[0], want[0], err_msg=f"{label} parent")
    np.testing.assert_allclose(got[2], want[2], rtol=1e-6, atol=0, err_msg=f"{label} joint")
    return got


CASES = [
    # (B, S, V, H, k, budget)
    (1, 1, 10, 0, 1, 1),
    (2, 3, 300, 60, 3, 16),
    (3, 4, 1000, 1000, 4, 40),          # every token hot
    (2, 5, 777, 0, 5, 100),             # no token information at all
    (4, 2, 4096, 512, 16, 256),         # largest branch number and budget
    (2, 16, 600, 100, 2, 33),           # most steps
    (5, 7, 5000, 1200, 8, 64),
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_tree_build_cases(oracle_mod, case):
    T = U.require_gpu()
    B, S, V, H, k, budget = CASES[case]
    x = W.make_tree_build_inputs(f"c{case}", 100 + case, B=B, S=S, V=V, H=H, k=k, budget=budget)
    compare(oracle_mod, T, x, f"case{case}")


def test_tree_build_narrative(oracle_mod):
    """The worked example of §5.2 (golden fixture) on the GPU."""
    T = U.require_gpu()
    from tests.test_oracle_tree_build import narrative
    g, ids, logits, table, hot = narrative()
    V = len(g["vocab"])
    hot_index = np.arange(V, dtype=np.int32)
    x = W.TreeBuildInputs("narrative", 1, logits.shape[1], V, V, g["k"], 11, logits,
                          np.array([ids[g["root"]]], np.int32), table, hot, hot_index)
    par, tok, jnt, nn = compare(oracle_mod, T, x, "narrative")
    names = [g["vocab"][t] for t in tok[0]]
    assert names[3] == "server" and jnt[0, 3] == pytest.approx(0.42, rel=1e-6)
    assert names[7] == "optimization" and jnt[0, 7] == pytest.approx(0.294, rel=1e-6)


def test_tree_build_full_vocabulary(oracle_mod):
    """The 8B-shaped vocabulary (128256) with a quarter of the hot table (8192
    hot tokens)."""
    T = U.require_gpu()
    x = W.make_tree_build_inputs("full", 7, B=4, S=7, V=128256, H=8192, k=8, budget=64)
    compare(oracle_mod, T, x, "full-vocab")


def test_tree_build_and_resample_bench_presets(oracle_mod):
    """The benchmarked workloads themselves, whole: 16 sequences, 7 steps,
    vocabulary 128256 with 32768 hot tokens, k 8, budget 64; then re-sampling
    on the same inputs with the benchmark's accept lengths and bonus tokens."""
    T = U.require_gpu()
    x = W.tree_build_preset("tb_llama8b_bs16")
    compare(oracle_mod, T, x, "tb_llama8b_bs16")
    bonus, alen = W.resample_inputs(x, 7)
    compare_resample(oracle_mod, T, x, bonus, alen, 1, "rs_llama8b_bs16-shapes")


def test_tree_build_feeds_verification(oracle_mod):
    """The builder's (parent, token, num_nodes) are valid tree inputs of the
    verification calls: a ragged accept over them matches the oracle."""
    T = U.require_gpu()
    x = W.make_tree_build_inputs("feed", 9, B=3, S=3, V=500, H=100, k=3, budget=20)
    par, tok, jnt, nn = run_gpu(T, x)
    assert (nn == 1 + 3 + 2 * 9).all() or (nn == 20).all()
    rng = np.random.default_rng(0)
    logits = rng.standard_normal((x.B, x.budget, x.V)).astype(np.float32)
    a, alen, aidx, bonus = T.tree_argmax_accept(U.dev(logits), U.dev(tok), U.dev(par),
                                                num_nodes=U.dev(nn))
    torch.cuda.synchronize()
    ra = oracle_mod.argmax(logits)
    rl, ri, rb = oracle_mod.accept(tok, par, ra, num_nodes=nn)
    np.testing.assert_array_equal(alen.cpu().numpy(), rl)
    np.testing.assert_array_equal(aidx.cpu().numpy(), ri)
    np.testing.assert_array_equal(bonus.cpu().numpy(), rb)


def test_tree_build_reuses_workspace(oracle_mod):
    """Two calls in a row on one workspace, the second smaller: nothing of the
    first call leaks into the second."""
    T = U.require_gpu()
    big = W.make_tree_build_inputs("big", 21, B=4, S=6, V=3000, H=700, k=6, budget=80)
    small = W.make_tree_build_inputs("small", 22, B=2, S=2, V=400, H=50, k=2, budget=9)
    ws = torch.empty(T.tree_build_workspace_size(4, 6, 3000, 700, 6), dtype=torch.uint8,
                     device="cuda")
    for x in (big, small):
        tab = U.dev(x.table.view(np.int16)).view(torch.bfloat16)
        par, tok, jnt, nn = T.tree_build(U.dev(x.logits), U.dev(x.root), tab, U.dev(x.hot_vocab),
                                         U.dev(x.hot_index), k=x.k, budget=x.budget, workspace=ws)
        torch.cuda.synchronize()
        want = oracle_mod.tree_build(x.logits, x.root, x.table, x.hot_vocab, x.k, x.budget)
        np.testing.assert_array_equal(tok.cpu().numpy(), want[1])
        np.testing.assert_array_equal(par.cpu().numpy(), want[0])
        np.testing.assert_array_equal(nn.cpu().numpy(), want[3])


def test_tree_build_workspace_alignment(oracle_mod):
    """Full expansion chunks load four columns per lane when the rows and the
    caller's arrays are aligned for it; a workspace that is only 8-byte aligned
    (the documented minimum), or a table and hot-id array one element off, take
    the narrow loads and build the same trees."""
    T = U.require_gpu()
    x = W.make_tree_build_inputs("align", 23, B=2, S=3, V=5000, H=4096, k=4, budget=30)
    n = T.tree_build_workspace_size(x.B, x.S, x.V, x.H, x.k)
    ws = torch.empty(n + 16, dtype=torch.uint8, device="cuda")
    margins = []
    want = oracle_mod.tree_build(x.logits, x.root, x.table, x.hot_vocab, x.k, x.budget, margins)
    assert min(margins) > 1e-9
    tab = U.dev(x.table.view(np.int16)).view(torch.bfloat16)
    got = []
    for off in (0, 8):
        print(f"case workspace offset {off}", flush=True)
        par, tok, jnt, nn = T.tree_build(U.dev(x.logits), U.dev(x.root), tab, U.dev(x.hot_vocab),
                                         U.dev(x.hot_index), k=x.k, budget=x.budget,
                                         workspace=ws[off:off + n])
        torch.cuda.synchronize()
        got.append((par.cpu().numpy(), tok.cpu().numpy(), jnt.cpu().numpy(), nn.cpu().numpy()))
        np.testing.assert_array_equal(got[-1][3], want[3])
        np.testing.assert_array_equal(got[-1][1], want[1])
        np.testing.assert_array_equal(got[-1][0], want[0])
        np.testing.assert_allclose(got[-1][2], want[2], rtol=1e-6, atol=0)
    for a, b in zip(got[0][:2] + got[0][3:], got[1][:2] + got[1][3:]):
        np.testing.assert_array_equal(a, b)
    # the caller's table and hot ids off the wide loads' alignment (one element
    # into a larger buffer): the narrow loads, the same trees
    print("case table and hot ids one element off", flush=True)
    tbuf = torch.empty(x.H * x.H + 1, dtype=torch.bfloat16, device="cuda")
    tbuf[1:].copy_(tab.reshape(-1))
    vbuf = torch.empty(x.H + 1, dtype=torch.int32, device="cuda")
    vbuf[1:].copy_(U.dev(x.hot_vocab))
    par, tok, jnt, nn = T.tree_build(U.dev(x.logits), U.dev(x.root), tbuf[1:].view(x.H, x.H),
                                     vbuf[1:], U.dev(x.hot_index), k=x.k, budget=x.budget,
                                     workspace=ws[:n])
    torch.cuda.synchronize()
    np.testing.assert_array_equal(nn.cpu().numpy(), want[3])
    np.testing.assert_array_equal(tok.cpu().numpy(), want[1])
    np.testing.assert_array_equal(par.cpu().numpy(), want[0])
    np.testing.assert_allclose(jnt.cpu().numpy(), want[2], rtol=1e-6, atol=0)


# ---------------------------------------------------------------- re-sampling (Alg. 2)
def run_resample(T, x, bonus, alen, r, budget=None, k=None):
    budget = x.budget if budget is None else budget
    k = x.k if k is None else k
    H = x.H
    tab = U.dev(x.table.view(np.int16)).view(torch.bfloat16) if H > 0 else None
    out = T.tree_resample(U.dev(x.logits), U.dev(bonus), U.dev(alen), tab,
                          U.dev(x.hot_vocab) if H > 0 else None,
                          U.dev(x.hot_index) if H > 0 else None, k=k, r=r, budget=budget)
    torch.cuda.synchronize()
    return [t.cpu().numpy() for t in out]


def compare_resample(oracle_mod, T, x, bonus, alen, r, label):
    print(f"case {label}: B={x.B} S={x.S} V={x.V} H={x.H} k={x.k} r={r} "
          f"accept_len={alen.tolist()}", flush=True)
    margins = []
    want = oracle_mod.resample(x.logits, bonus, alen, x.table, x.hot_vocab, x.k, r, x.budget,
                               margins)
    if margins:
        assert min(margins) > 1e-9, f"{label}: near-tie in the oracle ({min(margins):.2e})"
    got = run_resample(T, x, bonus, alen, r)
    np.testing.assert_array_equal(got[3], want[3], err_msg=f"{label} num_nodes")
    np.testing.assert_array_equal(got[1], want[1], err_msg=f"{label} token")
    np.testing.assert_array_equal(got[0], want[0], err_msg=f"{label} parent")
    np.testing.assert_allclose(got[2], want[2], rtol=1e-6, atol=0, err_msg=f"{label} joint")
    return got


@pytest.mark.parametrize("case", range(3))
def test_resample_cases(oracle_mod, case):
    T = U.require_gpu()
    B, S, V, H, k, budget, r = [(6, 5, 800, 200, 3, 30, 1), (8, 7, 5000, 1000, 8, 64, 2),
                                (4, 16, 600, 0, 2, 40, 0)][case]
    x = W.make_tree_build_inputs(f"rs{case}", 200 + case, B=B, S=S, V=V, H=H, k=k, budget=budget)
    rng = np.random.default_rng(case)
    alen = rng.integers(0, S + 2, B).astype(np.int32)         # 0 .. S+1, every window kind
    alen[0], alen[-1] = 1, S + 1
    bonus = rng.integers(0, V, B).astype(np.int32)
    if H:
        bonus[1::2] = x.hot_vocab[rng.integers(0, H, len(bonus[1::2]))]
    compare_resample(oracle_mod, T, x, bonus, alen, r, f"resample{case}")


def test_resample_narrative(oracle_mod):
    """The re-sampling narrative of §5.3 (golden fixture) on the GPU."""
    T = U.require_gpu()
    from tests.test_oracle_tree_build import resample_narrative
    g, ids, logits, table, hot = resample_narrative()
    V = len(g["vocab"])
    x = W.TreeBuildInputs("rs-narrative", 1, logits.shape[1], V, V, g["k"], 16, logits,
                          np.array([0], np.int32), table, hot, np.arange(V, dtype=np.int32))
    got = compare_resample(oracle_mod, T, x, np.array([ids[g["bonus"]]], np.int32),
                           np.array([g["accept_len"]], np.int32), g["r"], "rs-narrative")
    names = [g["vocab"][t] for t in got[1][0][:3]]
    assert names == ["quantization", "accuracy", "method"]


def test_speculative_iteration_chain(oracle_mod):
    """One speculative iteration end to end on the GPU, each stage checked
    against the oracle: build the draft trees, verify them (greedy accept over
    synthetic target logits with some drafts made acceptable), re-sample from
    the bonus tokens and accepted lengths."""
    T = U.require_gpu()
    x = W.make_tree_build_inputs("chain", 77, B=6, S=5, V=2000, H=400, k=3, budget=24)
    par, tok, jnt, nn = run_gpu(T, x)
    want = oracle_mod.tree_build(x.logits, x.root, x.table, x.hot_vocab, x.k, x.budget)
    np.testing.assert_array_equal(tok, want[1])
    rng = np.random.default_rng(3)
    tgt = rng.standard_normal((x.B, x.budget, x.V)).astype(np.float32)
    for b in range(x.B):                                   # let the target agree on a path
        depth = int(rng.integers(0, 4))
        i = 0
        for _ in range(depth):
            kids = [c for c in range(1, nn[b]) if par[b, c] == i]
            if not kids:
                break
            c = kids[int(rng.integers(0, len(kids)))]
            tgt[b, i, tok[b, c]] += 50.0
            i = c
    a, alen, aidx, bonus = T.tree_argmax_accept(U.dev(tgt), U.dev(tok), U.dev(par),
                                                num_nodes=U.dev(nn))
    torch.cuda.synchronize()
    alen, bonus = alen.cpu().numpy(), bonus.cpu().numpy()
    rl, ri, rb = oracle_mod.accept(tok, par, oracle_mod.argmax(tgt), num_nodes=nn)
    np.testing.assert_array_equal(alen, rl)
    np.testing.assert_array_equal(bonus, rb)
    print(f"accept_len {alen.tolist()}", flush=True)
    compare_resample(oracle_mod, T, x, bonus, alen, 1, "chain-resample")
