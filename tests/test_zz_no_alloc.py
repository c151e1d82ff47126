"""tree_argmax_accept_noalloc (static per-GPU scratch, no allocation) against
tree_argmax_accept (caller's workspace) and the oracle, through the C ABI: two
calls in a row on the same GPU, the second smaller, so the second call runs on
a scratch that still holds the first call's keys. Everything is bit-exact."""
import numpy as np
import pytest
import torch

from paper_2602_21224_amd import workloads as W
from tests import gpu_util as U

pytestmark = pytest.mark.gpu


def _outputs(B, N):
    mk = lambda *shape: torch.full(shape, -7, dtype=torch.int32, device="cuda")
    return dict(argmax_out=mk(B, N), accept_len=mk(B), accept_idx=mk(B, N), bonus_token=mk(B))


def test_noalloc_matches_workspace_call_twice(oracle_mod):
    T = U.require_gpu()
    big = W.preset("llama8b_bs16", boost_amount=20.0, boost_prob=1.0)
    rng = np.random.default_rng(17)
    B, N, V = 3, 10, 5000
    small_logits = rng.standard_normal((B, N, V), dtype=np.float32)
    small_parent = np.stack([W.tree_uniform_forest(rng, N) for _ in range(B)])
    small_draft = rng.integers(0, V, (B, N)).astype(np.int32)
    small_nn = np.array([10, 0, 4], np.int32)
    cases = [("llama8b_bs16+20", big.logits, big.draft, big.parent, None),
             ("small-ragged", small_logits, small_draft, small_parent, small_nn)]
    for label, logits, draft, parent, nn in cases:
        Bc, Nc, Vc = logits.shape
        print(f"case {label}: B={Bc} N={Nc} V={Vc}", flush=True)
        dl, dd, dp = U.dev(logits), U.dev(draft), U.dev(parent)
        dnn = None if nn is None else U.dev(nn)
        ref = T.tree_argmax_accept(dl, dd, dp, num_nodes=dnn)
        got = _outputs(Bc, Nc)
        T.tree_argmax_accept_noalloc(dl, dd, dp, num_nodes=dnn, **got)
        torch.cuda.synchronize()
        names = ("argmax_out", "accept_len", "accept_idx", "bonus_token")
        for name, r in zip(names, ref):
            assert torch.equal(got[name], r), f"{label}: {name} differs from the workspace call"
        ra = oracle_mod.argmax(logits)
        if nn is not None:
            ra = np.where(np.arange(Nc)[None, :] < nn[:, None], ra, -1)
        wl, wi, wb = oracle_mod.accept(draft, parent, ra, num_nodes=nn)
        np.testing.assert_array_equal(got["argmax_out"].cpu().numpy(), ra)
        np.testing.assert_array_equal(got["accept_len"].cpu().numpy(), wl)
        np.testing.assert_array_equal(got["accept_idx"].cpu().numpy(), wi)
        np.testing.assert_array_equal(got["bonus_token"].cpu().numpy(), wb)


def test_noalloc_rejects_batches_beyond_the_scratch():
    T = U.require_gpu()
    logits = torch.zeros((2048, 256, 1), dtype=torch.float32, device="cuda")
    idx = torch.zeros((2048, 256), dtype=torch.int32, device="cuda")
    out = _outputs(2048, 256)
    from paper_2602_21224_amd._lib import TreeVerifyError
    with pytest.raises(TreeVerifyError, match="status -7"):
        T.tree_argmax_accept_noalloc(logits, idx, idx - 1, **out)
    assert (out["accept_len"] == -7).all()          # nothing was launched
