"""CPU oracle for the tree-verification step (TEST INFRASTRUCTURE ONLY).

Only `tests/`, `__graft_entry__.smoke()` and the benchmark's `cpu_baseline`
leg may import this package. The GPU library never links, loads or calls it,
and it shares no code with the GPU library.

The verification arithmetic lives in `oracle.c` (plain C, fp64, OpenMP across
independent items); this module only compiles it with gcc and marshals numpy
arrays. Each wrapper cites the passage of the paper the C function follows.
The draft-tree builder (Alg. 1 with budget pruning) is `tree_build.py`, plain
numpy.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
# TREEVERIFY_ORACLE_LIB names a prebuilt oracle library to load instead (the
# sanitizer test builds one with AddressSanitizer and UBSan).
_LIB_OVERRIDE = os.environ.get("TREEVERIFY_ORACLE_LIB")
_LIB = _LIB_OVERRIDE or os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile oracle.c with gcc (fp64, no fast-math, no FMA contraction)."""
    if _LIB_OVERRIDE:
        return _LIB
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
               "-shared", "-fPIC", _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        lib = ctypes.CDLL(_LIB)
        p = ctypes.c_void_p
        i = ctypes.c_int
        lib.oracle_tree_attention.argtypes = [p] * 9 + [i] * 8 + [ctypes.c_double, p, p]
        lib.oracle_tree_attention.restype = i
        lib.oracle_tree_attention_rows.argtypes = [p] * 9 + [i] * 8 + [ctypes.c_double, p, i,
                                                                        p, p]
        lib.oracle_tree_attention_rows.restype = i
        lib.oracle_argmax.argtypes = [p, ctypes.c_long, ctypes.c_long, p]
        lib.oracle_argmax.restype = None
        lib.oracle_accept.argtypes = [p, p, p, p, i, i, p, p, p]
        lib.oracle_accept.restype = i
        lib.oracle_kv_compact.argtypes = [p] * 8 + [i] * 7
        lib.oracle_kv_compact.restype = i
        lib.oracle_num_threads.argtypes = []
        lib.oracle_num_threads.restype = i
        lib.oracle_set_num_threads.argtypes = [i]
        lib.oracle_set_num_threads.restype = None
        _lib = lib
    return _lib


def _ptr(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"], "oracle inputs must be C-contiguous"
    return a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def _opt(a, n):
    """Optional per-sequence int32 array of length n, or None."""
    if a is None:
        return None
    a = _c(a, np.int32).reshape(-1)
    if a.shape[0] != n:
        raise ValueError("num_nodes must hold one count per sequence")
    return a


def _optr(a):
    return None if a is None else _ptr(a)


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def set_num_threads(n: int) -> None:
    """Threads of the OpenMP loops from now on (results do not depend on it)."""
    _load().oracle_set_num_threads(int(n))


def tree_attention(q, k_tree, v_tree, k_cache, v_cache, page_table, kv_len, parent,
                   scale: float = 0.0, num_nodes=None):
    """Tree-masked attention (§2.1 tree-shaped verification mask; §8 SpecInfer
    masking; §1 attention over all cached keys). Inputs are bf16 bit arrays in
    the layouts of `paper_2602_21224_amd.workloads`. Returns (out, lse) as fp64
    arrays [B, N, Hq, D] and [B, N, Hq]. `num_nodes` [B] (optional) gives each
    sequence's node count, e.g. a verification-fusion forest (§6.2) padded to
    N; rows of the padding nodes are zeros with lse -inf."""
    q = _c(q, np.uint16)
    k_tree = _c(k_tree, np.uint16)
    v_tree = _c(v_tree, np.uint16)
    k_cache = _c(k_cache, np.uint16)
    v_cache = _c(v_cache, np.uint16)
    page_table = _c(page_table, np.int32)
    kv_len = _c(kv_len, np.int32)
    parent = _c(parent, np.int32)
    B, N, Hq, D = q.shape
    Hkv = k_tree.shape[2]
    num_pages, P = k_cache.shape[0], k_cache.shape[1]
    max_pages = page_table.shape[1]
    nn = _opt(num_nodes, B)
    out = np.zeros((B, N, Hq, D), dtype=np.float64)
    lse = np.zeros((B, N, Hq), dtype=np.float64)
    rc = _load().oracle_tree_attention(
        _ptr(q), _ptr(k_tree), _ptr(v_tree), _ptr(k_cache), _ptr(v_cache), _ptr(page_table),
        _ptr(kv_len), _ptr(parent), _optr(nn), B, N, Hq, Hkv, D, P, max_pages, num_pages,
        float(scale), _ptr(out), _ptr(lse))
    if rc == -2:
        raise MemoryError("oracle_tree_attention: scratch allocation failed")
    if rc != 0:
        raise ValueError("oracle_tree_attention rejected its arguments")
    return out, lse


def tree_attention_rows(q, k_tree, v_tree, k_cache, v_cache, page_table, kv_len, parent, items,
                        scale: float = 0.0, num_nodes=None):
    """The same attention for selected (b, i, h) rows only; items is an int
    array [n, 3]. Returns (out [n, D], lse [n]) in fp64."""
    q = _c(q, np.uint16)
    k_tree = _c(k_tree, np.uint16)
    v_tree = _c(v_tree, np.uint16)
    k_cache = _c(k_cache, np.uint16)
    v_cache = _c(v_cache, np.uint16)
    page_table = _c(page_table, np.int32)
    kv_len = _c(kv_len, np.int32)
    parent = _c(parent, np.int32)
    items = _c(items, np.int32).reshape(-1, 3)
    B, N, Hq, D = q.shape
    Hkv = k_tree.shape[2]
    num_pages, P = k_cache.shape[0], k_cache.shape[1]
    nn = _opt(num_nodes, B)
    out = np.zeros((len(items), D), dtype=np.float64)
    lse = np.zeros(len(items), dtype=np.float64)
    rc = _load().oracle_tree_attention_rows(
        _ptr(q), _ptr(k_tree), _ptr(v_tree), _ptr(k_cache), _ptr(v_cache), _ptr(page_table),
        _ptr(kv_len), _ptr(parent), _optr(nn), B, N, Hq, Hkv, D, P, page_table.shape[1], num_pages,
        float(scale), _ptr(items), len(items), _ptr(out), _ptr(lse))
    if rc == -2:
        raise MemoryError("oracle_tree_attention_rows: scratch allocation failed")
    if rc != 0:
        raise ValueError("oracle_tree_attention_rows rejected its arguments")
    return out, lse


def argmax(logits):
    """Per-row greedy argmax (§7.1 evaluates at temperature 0): lowest index of
    the maximum, -0 == +0, first NaN wins. logits [..., V] fp32 -> int32 [...]."""
    logits = _c(logits, np.float32)
    V = logits.shape[-1]
    rows = logits.size // V if V else 0
    out = np.zeros(logits.shape[:-1], dtype=np.int32)
    _load().oracle_argmax(_ptr(logits), rows, V, _ptr(out))
    return out


def accept(draft, parent, amax, num_nodes=None):
    """Greedy longest accepted path and bonus token (§5.3; Alg. 2's
    ground-truth token). Returns (accept_len [B], accept_idx [B, N], bonus [B]).
    With `num_nodes` only each sequence's first num_nodes[b] nodes take part;
    a sequence with none accepts nothing (length 0, bonus -1)."""
    draft = _c(draft, np.int32)
    parent = _c(parent, np.int32)
    amax = _c(amax, np.int32)
    B, N = parent.shape
    nn = _opt(num_nodes, B)
    alen = np.zeros(B, dtype=np.int32)
    aidx = np.zeros((B, N), dtype=np.int32)
    bonus = np.zeros(B, dtype=np.int32)
    rc = _load().oracle_accept(_ptr(draft), _ptr(parent), _ptr(amax), _optr(nn), B, N,
                               _ptr(alen), _ptr(aidx), _ptr(bonus))
    if rc == -2:
        raise MemoryError("oracle_accept: scratch allocation failed")
    if rc != 0:
        raise ValueError("oracle_accept: parent[i] must lie in [-1, i-1]")
    return alen, aidx, bonus


def kv_compact(k_tree, v_tree, k_cache, v_cache, page_table, kv_len, accept_idx, accept_len):
    """Copy the accepted path's K/V rows to cache positions kv_len .. kv_len +
    accept_len - 1 (§1 KV cache of committed tokens). Works on copies; returns
    the new (k_cache, v_cache)."""
    k_tree = _c(k_tree, np.uint16)
    v_tree = _c(v_tree, np.uint16)
    kc = np.array(k_cache, dtype=np.uint16, order="C", copy=True)
    vc = np.array(v_cache, dtype=np.uint16, order="C", copy=True)
    page_table = _c(page_table, np.int32)
    kv_len = _c(kv_len, np.int32)
    accept_idx = _c(accept_idx, np.int32)
    accept_len = _c(accept_len, np.int32)
    B, N, Hkv, D = k_tree.shape
    num_pages, P = kc.shape[0], kc.shape[1]
    rc = _load().oracle_kv_compact(_ptr(k_tree), _ptr(v_tree), _ptr(kc), _ptr(vc),
                                   _ptr(page_table), _ptr(kv_len), _ptr(accept_idx),
                                   _ptr(accept_len), B, N, Hkv, D, P, page_table.shape[1],
                                   num_pages)
    if rc != 0:
        raise ValueError("oracle_kv_compact: destination outside the page table or pool")
    return kc, vc


from .tree_build import resample, tree_build  # noqa: E402  (Alg. 1, Alg. 2, pruning; numpy)
from .lm_head import lm_head_argmax, lm_head_logits  # noqa: E402  (LM head + argmax; numpy)
