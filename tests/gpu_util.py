"""Helpers for the GPU parity tests: upload numpy workloads to device tensors
and compare against the oracle. Nothing here computes the method."""
from __future__ import annotations

import numpy as np
import pytest
import torch

ATOL = 2e-2      # attention tolerance for bf16 inputs, fp32 accumulation, bf16 output
RTOL = 1e-2


def require_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2602_21224_amd as T
    T.load()          # raises if the HIP library is missing: no fallback
    return T


def dev_bf16(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()


def dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def bf16_to_f64(t: torch.Tensor) -> np.ndarray:
    return t.float().cpu().numpy().astype(np.float64)


def upload(w):
    return dict(q=dev_bf16(w.q), k_tree=dev_bf16(w.k_tree), v_tree=dev_bf16(w.v_tree),
                k_cache=dev_bf16(w.k_cache), v_cache=dev_bf16(w.v_cache),
                page_table=dev(w.page_table), kv_len=dev(w.kv_len), parent=dev(w.parent),
                num_nodes=None if w.num_nodes is None else dev(w.num_nodes))


def gpu_attention(T, w, scale=0.0, d=None):
    d = d or upload(w)
    out, lse = T.tree_verify_attention(d["q"], d["k_tree"], d["v_tree"], d["k_cache"],
                                       d["v_cache"], d["page_table"], d["kv_len"], d["parent"],
                                       max_kv_len=w.max_kv_len, scale=scale,
                                       num_nodes=d["num_nodes"])
    torch.cuda.synchronize()
    return bf16_to_f64(out), lse.cpu().numpy().astype(np.float64)


def assert_attention_close(got, want, lse_got=None, lse_want=None, label=""):
    err = np.abs(got - want)
    bound = ATOL + RTOL * np.abs(want)
    bad = err > bound
    print(f"[{label}] max abs err {err.max():.3e}, mean {err.mean():.3e}", flush=True)
    assert not bad.any(), (f"{label}: {bad.sum()} of {bad.size} outside tolerance; "
                           f"max err {err.max():.3e}")
    # Rounding P to bf16 perturbs each weight by up to 2^-9, so a single output can
    # be off by about 2^-9 * max|v| over its visible keys; the mean error is a much
    # tighter bug signal (a dropped or extra key moves it by orders of magnitude).
    assert err.mean() <= 2e-3, f"{label}: mean error {err.mean():.3e}"
    if lse_got is not None:
        lerr = np.abs(lse_got - lse_want)
        print(f"[{label}] lse max abs err {lerr.max():.3e}", flush=True)
        assert np.all(lerr <= 2e-3 + 1e-4 * np.abs(lse_want)), f"{label}: lse error {lerr.max()}"
