"""GPU parity of tree_lm_head_argmax_accept (the LM head fused with greedy
verification) against the CPU oracle, through the C ABI.

The kernel sums bf16 products in fp32 on the matrix cores, the oracle sums
them exactly (fp64). Any fp32 summation order puts a computed logit within
gamma_d * sum_i |h_i w_vi| of the exact one (gamma_d = d u / (1 - d u),
u = 2^-24; the products themselves are exact in fp32), and
sum_i |h_i w_vi| <= sum_i |h_i| * max|W| =: S_r for every v. So:
  * rows whose exact top-2 margin exceeds 2 gamma_d S_r have one correct
    answer and must match the oracle's argmax exactly;
  * on the other rows several entries are correct fp32 argmaxes: the GPU's
    pick must be a valid vocabulary id whose exact logit lies within
    2 gamma_d S_r of the exact maximum.
Acceptance (accept_len, accept_idx, bonus) is checked bit-exactly against the
oracle's acceptance applied to the argmax the GPU produced."""
import numpy as np
import pytest
import torch

from paper_2602_21224_amd import workloads as W
from tests import gpu_util as U

pytestmark = pytest.mark.gpu


def gamma(d):
    u = 2.0 ** -24
    return d * u / (1 - d * u)


def upload(x):
    return (U.dev_bf16(x.hidden), U.dev_bf16(x.w_head), U.dev(x.draft), U.dev(x.parent),
            None if x.num_nodes is None else U.dev(x.num_nodes))


def run_gpu(T, x, ws=None):
    hid, w, draft, par, nn = upload(x)
    out = T.tree_lm_head_argmax_accept(hid, w, draft, par, num_nodes=nn, workspace=ws)
    torch.cuda.synchronize()
    return [t.cpu().numpy() for t in out]


def real_rows(x):
    counts = np.full(x.B, x.N) if x.num_nodes is None else np.clip(x.num_nodes, 0, x.N)
    return np.array([b * x.N + i for b in range(x.B) for i in range(int(counts[b]))], np.int64)


def check_argmax(oracle_mod, x, got_amax, rows, label, min_decisive=0.5):
    """Check the GPU's argmax of the given flat rows (see the module docstring)."""
    hid = x.hidden.reshape(-1, x.d)[rows]
    got = got_amax.reshape(-1)[rows]
    want, margin, _ = oracle_mod.lm_head_argmax(hid, x.w_head)
    h = W.bf16_bits_to_f32(hid).astype(np.float64)
    wmax = float(np.abs(W.bf16_bits_to_f32(x.w_head)).max())
    bound = gamma(x.d) * np.abs(h).sum(1) * wmax
    decisive = margin > 2 * bound
    print(f"[{label}] {len(rows)} rows, {decisive.sum()} decisive", flush=True)
    assert decisive.mean() >= min_decisive, f"{label}: too few decisive rows for a parity check"
    np.testing.assert_array_equal(got[decisive], want[decisive], err_msg=f"{label} argmax")
    assert ((got >= 0) & (got < x.V)).all(), f"{label}: argmax out of range"
    for j in np.nonzero(~decisive)[0]:
        wg = W.bf16_bits_to_f32(x.w_head[got[j]]).astype(np.float64)
        ww = W.bf16_bits_to_f32(x.w_head[want[j]]).astype(np.float64)
        assert h[j] @ wg >= h[j] @ ww - 2 * bound[j], f"{label}: row {rows[j]} picked a non-maximum"


def check_accept(oracle_mod, x, got, label):
    amax, alen, aidx, bonus = got
    padding = np.ones(x.B * x.N, bool)
    padding[real_rows(x)] = False
    assert (amax.reshape(-1)[padding] == -1).all(), f"{label}: padding rows got an argmax"
    rl, ri, rb = oracle_mod.accept(x.draft, x.parent, amax, num_nodes=x.num_nodes)
    np.testing.assert_array_equal(alen, rl, err_msg=f"{label} accept_len")
    np.testing.assert_array_equal(aidx, ri, err_msg=f"{label} accept_idx")
    np.testing.assert_array_equal(bonus, rb, err_msg=f"{label} bonus")


CASES = [
    # (B, N, V, d, num_nodes)
    (2, 16, 1000, 256, None),
    (3, 37, 1000, 192, [37, 5, 20]),     # ragged rows and vocabulary, three K units
    (1, 8, 257, 64, None),               # one K unit, one entry past a vocabulary tile
    (2, 4, 300, 128, None),              # two K units
    (1, 3, 1, 128, None),                # a single vocabulary entry
    (4, 64, 20000, 1024, None),          # full row tile, many vocabulary tiles
    (5, 64, 3000, 512, [64, 0, 17, 64, 1]),   # row tiles split across sequences, empty ones
    (6, 64, 900, 320, None),             # two row blocks, five K units: a rotated group of four + one
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_lm_head_cases(oracle_mod, case):
    T = U.require_gpu()
    B, N, V, d, nn = CASES[case]
    print(f"case lm{case}: B={B} N={N} V={V} d={d} num_nodes={nn}", flush=True)
    x = W.make_lm_head_inputs(f"lm{case}", 300 + case, B=B, N=N, V=V, d=d, num_nodes=nn)
    got = run_gpu(T, x)
    rows = real_rows(x)
    if len(rows):
        check_argmax(oracle_mod, x, got[0], rows, f"lm{case}",
                     min_decisive=0.0 if V == 1 else 0.5)
    check_accept(oracle_mod, x, got, f"lm{case}")


def test_lm_head_full_size_row_block(oracle_mod):
    """The 8B-shaped head (vocabulary 128256, hidden size 4096, 16 x 64 nodes)
    in the launch configuration the benchmark times; the oracle checks one
    complete 256-row tile block (rows 512..767, sequences 8..11) over the whole
    vocabulary, the acceptance all 1024 rows."""
    T = U.require_gpu()
    print("case lm_llama8b_bs16 (row block 2 of 4)", flush=True)
    x = W.lm_head_preset("lm_llama8b_bs16")
    got = run_gpu(T, x)
    rows = np.arange(512, 768)
    check_argmax(oracle_mod, x, got[0], rows, "lm_llama8b_bs16")
    check_accept(oracle_mod, x, got, "lm_llama8b_bs16")
    assert (got[1] > 1).sum() >= 4, "planted drafts should be accepted somewhere"


def test_lm_head_equal_rows_pick_lowest_id(oracle_mod):
    """Two identical head rows give bit-identical sums (same operands, same
    accumulation order), so the lower id must win, as in the definition."""
    T = U.require_gpu()
    x = W.make_lm_head_inputs("ties", 310, B=2, N=16, V=3000, d=512)
    want, _, _ = oracle_mod.lm_head_argmax(x.hidden.reshape(-1, x.d), x.w_head)
    r = 3
    win = int(want[r])
    low = 7 if win != 7 else 8
    x.w_head[low] = x.w_head[win]          # an earlier duplicate of row r's winner
    got = run_gpu(T, x)
    assert got[0].reshape(-1)[r] == min(low, win)


def test_lm_head_nan_column_wins():
    """A NaN anywhere in head row v makes every logit of column v NaN, and NaN
    counts as the maximum (first NaN on ties), so every node's argmax is v."""
    T = U.require_gpu()
    x = W.make_lm_head_inputs("nan", 311, B=2, N=8, V=700, d=128)
    x.w_head[600, 17] = W.BF16_NAN
    x.w_head[650, 3] = W.BF16_NAN
    got = run_gpu(T, x)
    assert (got[0] == 600).all()


def test_lm_head_reuses_workspace(oracle_mod):
    """Two calls in a row on one workspace, the second smaller: the row keys
    are reset by each call."""
    T = U.require_gpu()
    big = W.make_lm_head_inputs("big", 312, B=4, N=64, V=2000, d=256)
    small = W.make_lm_head_inputs("small", 313, B=1, N=10, V=500, d=64)
    ws = torch.empty(T.lm_head_workspace_size(4, 64, 2000, 256), dtype=torch.uint8, device="cuda")
    for x in (big, small):
        got = run_gpu(T, x, ws)
        check_argmax(oracle_mod, x, got[0], real_rows(x), x.name)
        check_accept(oracle_mod, x, got, x.name)


def test_lm_head_matches_unfused_path(oracle_mod):
    """Fused and unfused verification agree: logits computed by torch (bf16
    inputs, fp32 result) fed to tree_argmax_accept give the same acceptance
    wherever the rows are decisive."""
    T = U.require_gpu()
    x = W.make_lm_head_inputs("unfused", 314, B=4, N=64, V=5000, d=1024)
    hid, w, draft, par, _ = upload(x)
    fused = T.tree_lm_head_argmax_accept(hid, w, draft, par)
    logits = (hid.float().reshape(-1, x.d) @ w.float().t().contiguous()).reshape(x.B, x.N, x.V)
    unfused = T.tree_argmax_accept(logits.contiguous(), draft, par)
    torch.cuda.synchronize()
    want, margin, _ = oracle_mod.lm_head_argmax(x.hidden.reshape(-1, x.d), x.w_head)
    h = W.bf16_bits_to_f32(x.hidden.reshape(-1, x.d)).astype(np.float64)
    bound = gamma(x.d) * np.abs(h).sum(1) * float(np.abs(W.bf16_bits_to_f32(x.w_head)).max())
    dec = margin > 2 * bound
    fa, ua = fused[0].cpu().numpy().reshape(-1), unfused[0].cpu().numpy().reshape(-1)
    np.testing.assert_array_equal(fa[dec], ua[dec])
    np.testing.assert_array_equal(fa[dec], want[dec])
