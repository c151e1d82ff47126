"""ctypes binding of libtreeverify (argument marshalling only).

Each wrapper takes torch tensors that already live on the GPU, checks dtype,
shape and contiguity, and passes raw device pointers plus the current HIP
stream to the C entry point of the same name. Every step of the computation
runs in the library's HIP kernels; there is no fallback of any kind: if the
library is missing or a call returns an error status, a Python exception is
raised.
"""
from __future__ import annotations

import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
# TREEVERIFY_LIB names another build of the same library to load (the
# sanitizer test loads one whose host code carries AddressSanitizer and UBSan).
LIB_PATH = os.environ.get("TREEVERIFY_LIB") or os.path.join(HERE, "libtreeverify.so")

_lib = None


class TreeVerifyError(RuntimeError):
    pass


def load():
    """Load libtreeverify.so (built in-tree by `paper_2602_21224_amd.build`)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise TreeVerifyError(f"{LIB_PATH} is missing: build it with "
                              "`python -m paper_2602_21224_amd.build` (hipcc, gfx950)")
    lib = ctypes.CDLL(LIB_PATH)
    p, i, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
    lib.tv_abi_version.argtypes = []
    lib.tv_abi_version.restype = i
    lib.tv_status_string.argtypes = [i]
    lib.tv_status_string.restype = ctypes.c_char_p
    lib.tv_attention_workspace_size.argtypes = [i] * 5
    lib.tv_attention_workspace_size.restype = sz
    lib.tree_verify_attention.argtypes = [p] * 9 + [i] * 9 + [ctypes.c_float, p, p, p, sz, p]
    lib.tree_verify_attention.restype = i
    lib.tv_argmax_workspace_size.argtypes = [i] * 3
    lib.tv_argmax_workspace_size.restype = sz
    lib.tree_argmax_accept.argtypes = [p] * 4 + [i] * 3 + [p] * 5 + [sz, p]
    lib.tree_argmax_accept.restype = i
    lib.tree_argmax_accept_noalloc.argtypes = [p] * 4 + [i] * 3 + [p] * 5
    lib.tree_argmax_accept_noalloc.restype = i
    lib.kv_compact_accepted.argtypes = [p] * 8 + [i] * 7 + [p]
    lib.kv_compact_accepted.restype = i
    lib.tv_validate_inputs.argtypes = [p] * 4 + [i] * 5 + [p, p]
    lib.tv_validate_inputs.restype = i
    lib.tv_tree_build_workspace_size.argtypes = [i] * 5
    lib.tv_tree_build_workspace_size.restype = sz
    lib.tree_build.argtypes = [p] * 5 + [i] * 6 + [p] * 5 + [sz, p]
    lib.tree_build.restype = i
    lib.tree_resample.argtypes = [p] * 6 + [i] * 7 + [p] * 5 + [sz, p]
    lib.tree_resample.restype = i
    lib.tv_lm_head_workspace_size.argtypes = [i] * 4
    lib.tv_lm_head_workspace_size.restype = sz
    lib.tree_lm_head_argmax_accept.argtypes = [p] * 5 + [i] * 4 + [p] * 5 + [sz, p]
    lib.tree_lm_head_argmax_accept.restype = i
    _lib = lib
    return lib


def _check(status: int, what: str):
    if status != 0:
        msg = load().tv_status_string(status).decode()
        raise TreeVerifyError(f"{what}: status {status} ({msg})")


def _ptr(t):
    return ctypes.c_void_p(0) if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


_BF16 = (torch.bfloat16, torch.int16, torch.uint16)


def _want(t, name, dtypes, shape=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be on the GPU")
    if t.dtype not in dtypes:
        raise TypeError(f"{name} has dtype {t.dtype}, expected one of {dtypes}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")


def abi_version() -> int:
    return int(load().tv_abi_version())


def attention_workspace_size(B, N, Hq, Hkv, D) -> int:
    return int(load().tv_attention_workspace_size(B, N, Hq, Hkv, D))


def argmax_workspace_size(B, N, V) -> int:
    return int(load().tv_argmax_workspace_size(B, N, V))


def tree_verify_attention(q, k_tree, v_tree, k_cache, v_cache, page_table, kv_len, parent, *,
                          max_kv_len: int, num_nodes=None, scale: float = 0.0, out=None,
                          lse=None, want_lse: bool = True, workspace=None, stream=None):
    """Tree-masked attention of every node over its sequence's paged prefix and
    its own root path. `num_nodes` (int32 [B], optional) makes the batch ragged.
    Returns (out bf16 [B,N,Hq,D], lse fp32 [B,N,Hq] or None)."""
    B, N, Hq, D = q.shape
    Hkv = k_tree.shape[2]
    num_pages, P = k_cache.shape[0], k_cache.shape[1]
    max_pages = page_table.shape[1]
    _want(q, "q", _BF16)
    _want(k_tree, "k_tree", _BF16, (B, N, Hkv, D))
    _want(v_tree, "v_tree", _BF16, (B, N, Hkv, D))
    _want(k_cache, "k_cache", _BF16, (num_pages, P, Hkv, D))
    _want(v_cache, "v_cache", _BF16, (num_pages, P, Hkv, D))
    _want(page_table, "page_table", (torch.int32,), (B, max_pages))
    _want(kv_len, "kv_len", (torch.int32,), (B,))
    _want(parent, "parent", (torch.int32,), (B, N))
    if num_nodes is not None:
        _want(num_nodes, "num_nodes", (torch.int32,), (B,))
    if out is None:
        out = torch.empty((B, N, Hq, D), dtype=torch.bfloat16, device=q.device)
    _want(out, "out", _BF16, (B, N, Hq, D))
    if lse is None and want_lse:
        lse = torch.empty((B, N, Hq), dtype=torch.float32, device=q.device)
    if lse is not None:
        _want(lse, "lse", (torch.float32,), (B, N, Hq))
    need = attention_workspace_size(B, N, Hq, Hkv, D)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=q.device)
    _want(workspace, "workspace", (torch.uint8,))
    st = load().tree_verify_attention(
        _ptr(q), _ptr(k_tree), _ptr(v_tree), _ptr(k_cache), _ptr(v_cache), _ptr(page_table),
        _ptr(kv_len), _ptr(parent), _ptr(num_nodes), B, N, Hq, Hkv, D, P, max_pages, num_pages,
        int(max_kv_len),
        float(scale), _ptr(out), _ptr(lse), _ptr(workspace), workspace.numel(), _stream(stream))
    _check(st, "tree_verify_attention")
    return out, lse


def tree_argmax_accept(logits, draft_tokens, parent, *, num_nodes=None, argmax_out=None,
                       accept_len=None, accept_idx=None, bonus_token=None, workspace=None,
                       stream=None):
    """Per-node argmax, greedy longest accepted path and bonus token.
    `num_nodes` (int32 [B], optional) makes the batch ragged.
    Returns (argmax [B,N], accept_len [B], accept_idx [B,N], bonus [B]) int32."""
    B, N, V = logits.shape
    dev = logits.device
    _want(logits, "logits", (torch.float32,))
    _want(draft_tokens, "draft_tokens", (torch.int32,), (B, N))
    _want(parent, "parent", (torch.int32,), (B, N))
    if num_nodes is not None:
        _want(num_nodes, "num_nodes", (torch.int32,), (B,))
    mk = lambda shape: torch.empty(shape, dtype=torch.int32, device=dev)
    argmax_out = mk((B, N)) if argmax_out is None else argmax_out
    accept_len = mk((B,)) if accept_len is None else accept_len
    accept_idx = mk((B, N)) if accept_idx is None else accept_idx
    bonus_token = mk((B,)) if bonus_token is None else bonus_token
    for t, n, s in ((argmax_out, "argmax_out", (B, N)), (accept_len, "accept_len", (B,)),
                    (accept_idx, "accept_idx", (B, N)), (bonus_token, "bonus_token", (B,))):
        _want(t, n, (torch.int32,), s)
    need = argmax_workspace_size(B, N, V)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=dev)
    _want(workspace, "workspace", (torch.uint8,))
    st = load().tree_argmax_accept(
        _ptr(logits), _ptr(draft_tokens), _ptr(parent), _ptr(num_nodes), B, N, V, _ptr(argmax_out),
        _ptr(accept_len), _ptr(accept_idx), _ptr(bonus_token), _ptr(workspace),
        workspace.numel(), _stream(stream))
    _check(st, "tree_argmax_accept")
    return argmax_out, accept_len, accept_idx, bonus_token


def tree_argmax_accept_noalloc(logits, draft_tokens, parent, *, argmax_out, accept_len,
                               accept_idx, bonus_token, num_nodes=None, stream=None):
    """tree_argmax_accept with the library's static per-GPU scratch instead of a
    workspace: nothing is allocated, so every output tensor must be given.
    Calls that can overlap on one GPU race on that scratch."""
    B, N, V = logits.shape
    _want(logits, "logits", (torch.float32,))
    _want(draft_tokens, "draft_tokens", (torch.int32,), (B, N))
    _want(parent, "parent", (torch.int32,), (B, N))
    if num_nodes is not None:
        _want(num_nodes, "num_nodes", (torch.int32,), (B,))
    for t, n, s in ((argmax_out, "argmax_out", (B, N)), (accept_len, "accept_len", (B,)),
                    (accept_idx, "accept_idx", (B, N)), (bonus_token, "bonus_token", (B,))):
        _want(t, n, (torch.int32,), s)
    st = load().tree_argmax_accept_noalloc(
        _ptr(logits), _ptr(draft_tokens), _ptr(parent), _ptr(num_nodes), B, N, V,
        _ptr(argmax_out), _ptr(accept_len), _ptr(accept_idx), _ptr(bonus_token), _stream(stream))
    _check(st, "tree_argmax_accept_noalloc")
    return argmax_out, accept_len, accept_idx, bonus_token


def lm_head_workspace_size(B, N, V, d) -> int:
    return int(load().tv_lm_head_workspace_size(B, N, V, d))


def tree_lm_head_argmax_accept(hidden, w_head, draft_tokens, parent, *, num_nodes=None,
                               argmax_out=None, accept_len=None, accept_idx=None,
                               bonus_token=None, workspace=None, stream=None):
    """LM head fused with greedy verification: hidden [B,N,d] bf16 times
    w_head [V,d] bf16, per-node argmax of the product (never stored), then the
    acceptance of tree_argmax_accept.
    Returns (argmax [B,N], accept_len [B], accept_idx [B,N], bonus [B]) int32."""
    B, N, d = hidden.shape
    V = w_head.shape[0]
    dev = hidden.device
    _want(hidden, "hidden", _BF16)
    _want(w_head, "w_head", _BF16, (V, d))
    _want(draft_tokens, "draft_tokens", (torch.int32,), (B, N))
    _want(parent, "parent", (torch.int32,), (B, N))
    if num_nodes is not None:
        _want(num_nodes, "num_nodes", (torch.int32,), (B,))
    mk = lambda shape: torch.empty(shape, dtype=torch.int32, device=dev)
    argmax_out = mk((B, N)) if argmax_out is None else argmax_out
    accept_len = mk((B,)) if accept_len is None else accept_len
    accept_idx = mk((B, N)) if accept_idx is None else accept_idx
    bonus_token = mk((B,)) if bonus_token is None else bonus_token
    for t, n, s in ((argmax_out, "argmax_out", (B, N)), (accept_len, "accept_len", (B,)),
                    (accept_idx, "accept_idx", (B, N)), (bonus_token, "bonus_token", (B,))):
        _want(t, n, (torch.int32,), s)
    need = lm_head_workspace_size(B, N, V, d)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=dev)
    _want(workspace, "workspace", (torch.uint8,))
    st = load().tree_lm_head_argmax_accept(
        _ptr(hidden), _ptr(w_head), _ptr(draft_tokens), _ptr(parent), _ptr(num_nodes), B, N, V,
        d, _ptr(argmax_out), _ptr(accept_len), _ptr(accept_idx), _ptr(bonus_token),
        _ptr(workspace), workspace.numel(), _stream(stream))
    _check(st, "tree_lm_head_argmax_accept")
    return argmax_out, accept_len, accept_idx, bonus_token


def kv_compact_accepted(k_tree, v_tree, k_cache, v_cache, page_table, kv_len, accept_idx,
                        accept_len, *, stream=None):
    """Write the accepted path's K/V rows into the cache after each prefix (in place)."""
    B, N, Hkv, D = k_tree.shape
    num_pages, P = k_cache.shape[0], k_cache.shape[1]
    max_pages = page_table.shape[1]
    _want(k_tree, "k_tree", _BF16)
    _want(v_tree, "v_tree", _BF16, (B, N, Hkv, D))
    _want(k_cache, "k_cache", _BF16, (num_pages, P, Hkv, D))
    _want(v_cache, "v_cache", _BF16, (num_pages, P, Hkv, D))
    _want(page_table, "page_table", (torch.int32,), (B, max_pages))
    _want(kv_len, "kv_len", (torch.int32,), (B,))
    _want(accept_idx, "accept_idx", (torch.int32,), (B, N))
    _want(accept_len, "accept_len", (torch.int32,), (B,))
    st = load().kv_compact_accepted(
        _ptr(k_tree), _ptr(v_tree), _ptr(k_cache), _ptr(v_cache), _ptr(page_table), _ptr(kv_len),
        _ptr(accept_idx), _ptr(accept_len), B, N, Hkv, D, P, max_pages, num_pages,
        _stream(stream))
    _check(st, "kv_compact_accepted")
    return k_cache, v_cache


def tv_validate_inputs(page_table, kv_len, parent, *, P: int, num_pages: int, num_nodes=None,
                       stream=None):
    """Device-side contract check; returns the status bit set as a 1-element int32 tensor."""
    B, N = parent.shape
    max_pages = page_table.shape[1]
    _want(page_table, "page_table", (torch.int32,), (B, max_pages))
    _want(kv_len, "kv_len", (torch.int32,), (B,))
    _want(parent, "parent", (torch.int32,), (B, N))
    if num_nodes is not None:
        _want(num_nodes, "num_nodes", (torch.int32,), (B,))
    word = torch.empty(1, dtype=torch.int32, device=parent.device)
    st = load().tv_validate_inputs(_ptr(page_table), _ptr(kv_len), _ptr(parent), _ptr(num_nodes), B, N, P,
                                   max_pages, num_pages, _ptr(word), _stream(stream))
    _check(st, "tv_validate_inputs")
    return word


def tree_build_workspace_size(B, S, V, H, k) -> int:
    return int(load().tv_tree_build_workspace_size(B, S, V, H, k))


def tree_build(logits, root_token, token_info, hot_vocab, hot_index, *, k: int, budget: int,
               parent=None, token=None, joint=None, num_nodes=None, workspace=None, stream=None):
    """Draft tree by token-info sampling (Alg. 1) pruned to `budget` nodes (§5.2).

    logits [B, S, V] fp32, root_token [B] int32, token_info [H, H] bf16 (or
    None with H = 0), hot_vocab [H] and hot_index [V] int32. Returns (parent,
    token, joint, num_nodes): [B, budget] int32, int32, fp32 and [B] int32.
    """
    B, S, V = logits.shape
    _want(logits, "logits", (torch.float32,))
    _want(root_token, "root_token", (torch.int32,), (B,))
    H = 0 if token_info is None else token_info.shape[0]
    if H > 0:
        _want(token_info, "token_info", _BF16, (H, H))
        _want(hot_vocab, "hot_vocab", (torch.int32,), (H,))
        _want(hot_index, "hot_index", (torch.int32,), (V,))
    dev = logits.device
    mk = lambda shape, dt: torch.empty(shape, dtype=dt, device=dev)
    parent = mk((B, budget), torch.int32) if parent is None else parent
    token = mk((B, budget), torch.int32) if token is None else token
    joint = mk((B, budget), torch.float32) if joint is None else joint
    num_nodes = mk((B,), torch.int32) if num_nodes is None else num_nodes
    _want(parent, "parent", (torch.int32,), (B, budget))
    _want(token, "token", (torch.int32,), (B, budget))
    _want(joint, "joint", (torch.float32,), (B, budget))
    _want(num_nodes, "num_nodes", (torch.int32,), (B,))
    need = tree_build_workspace_size(B, S, V, H, k)
    if need == 0:
        raise TreeVerifyError(f"tree_build: unsupported shape B={B} S={S} V={V} H={H} k={k}")
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    st = load().tree_build(
        _ptr(logits), _ptr(root_token), _ptr(token_info if H > 0 else None),
        _ptr(hot_vocab if H > 0 else None), _ptr(hot_index if H > 0 else None), B, S, V, H, k,
        budget, _ptr(parent), _ptr(token), _ptr(joint), _ptr(num_nodes), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream))
    _check(st, "tree_build")
    return parent, token, joint, num_nodes


def tree_resample(logits, bonus_token, accept_len, token_info, hot_vocab, hot_index, *, k: int,
                  r: int, budget: int, parent=None, token=None, joint=None, num_nodes=None,
                  workspace=None, stream=None):
    """Re-sampled draft trees after verification (Alg. 2): rooted at the bonus
    tokens, drawn from logits rows accept_len .. S-1 when more than r remain.
    Same tensors and outputs as tree_build, plus bonus_token / accept_len [B]."""
    B, S, V = logits.shape
    _want(logits, "logits", (torch.float32,))
    _want(bonus_token, "bonus_token", (torch.int32,), (B,))
    _want(accept_len, "accept_len", (torch.int32,), (B,))
    H = 0 if token_info is None else token_info.shape[0]
    if H > 0:
        _want(token_info, "token_info", _BF16, (H, H))
        _want(hot_vocab, "hot_vocab", (torch.int32,), (H,))
        _want(hot_index, "hot_index", (torch.int32,), (V,))
    dev = logits.device
    mk = lambda shape, dt: torch.empty(shape, dtype=dt, device=dev)
    parent = mk((B, budget), torch.int32) if parent is None else parent
    token = mk((B, budget), torch.int32) if token is None else token
    joint = mk((B, budget), torch.float32) if joint is None else joint
    num_nodes = mk((B,), torch.int32) if num_nodes is None else num_nodes
    _want(parent, "parent", (torch.int32,), (B, budget))
    _want(token, "token", (torch.int32,), (B, budget))
    _want(joint, "joint", (torch.float32,), (B, budget))
    _want(num_nodes, "num_nodes", (torch.int32,), (B,))
    need = tree_build_workspace_size(B, S, V, H, k)
    if need == 0:
        raise TreeVerifyError(f"tree_resample: unsupported shape B={B} S={S} V={V} H={H} k={k}")
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    st = load().tree_resample(
        _ptr(logits), _ptr(bonus_token), _ptr(accept_len), _ptr(token_info if H > 0 else None),
        _ptr(hot_vocab if H > 0 else None), _ptr(hot_index if H > 0 else None), B, S, V, H, k, r,
        budget, _ptr(parent), _ptr(token), _ptr(joint), _ptr(num_nodes), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream))
    _check(st, "tree_resample")
    return parent, token, joint, num_nodes

