"""Host-side checks of the C ABI (CPU only; no kernel is ever launched).

The library loads, exports every function its header declares, and rejects
malformed arguments on the host with the documented status before touching
the device."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "treeverify.h")


@pytest.fixture(scope="module")
def lib():
    from paper_2602_21224_amd import _lib
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2602_21224_amd import build
        build.build()
    return _lib.load()


def declared():
    text = open(HEADER).read()
    return re.findall(r"TV_API\s+[\w\s\*]+?\b(\w+)\s*\(", text)


def test_header_declares_the_three_calls():
    names = set(declared())
    assert {"tree_verify_attention", "tree_argmax_accept", "kv_compact_accepted"} <= names


def test_every_declared_symbol_is_exported(lib):
    for name in declared():
        assert hasattr(lib, name), name


def test_only_declared_symbols_are_exported():
    import subprocess
    from paper_2602_21224_amd import _lib
    out = subprocess.run(["nm", "-D", "--defined-only", _lib.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = {l.split()[-1] for l in out.splitlines() if l.split()[1] == "T"}
    assert exported == set(declared())


def test_status_strings(lib):
    assert lib.tv_abi_version() == 5
    for code in range(0, -8, -1):
        assert lib.tv_status_string(code)
    assert lib.tv_status_string(-99) == b"unknown status"


FAKE = ctypes.c_void_p(0x10000)          # never dereferenced: checks return first
NULL = ctypes.c_void_p(0)
STREAM = ctypes.c_void_p(0)


def attn(lib, **kw):
    a = dict(q=FAKE, k_tree=FAKE, v_tree=FAKE, k_cache=FAKE, v_cache=FAKE, page_table=FAKE,
             kv_len=FAKE, parent=FAKE, num_nodes=NULL, B=2, N=8, Hq=8, Hkv=2, D=128, P=16,
             max_pages=4,
             num_pages=8, max_kv_len=32, scale=0.0, out=FAKE, lse=NULL, ws=FAKE,
             ws_bytes=1 << 40)
    a.update(kw)
    return lib.tree_verify_attention(*a.values(), STREAM)


def test_attention_argument_checks(lib):
    assert attn(lib, B=0) == 0
    assert attn(lib, q=NULL) == -1
    assert attn(lib, ws=NULL) == -1
    assert attn(lib, D=96) == -2
    assert attn(lib, N=0) == -2 and attn(lib, N=257) == -2
    assert attn(lib, Hq=6, Hkv=4) == -2
    assert attn(lib, P=12) == -2
    assert attn(lib, Hq=64, Hkv=2, N=128) == -2          # more than 2048 rows per KV head
    assert attn(lib, B=5000) == -2
    assert attn(lib, q=ctypes.c_void_p(0x10008)) == -3
    # well-formed on a machine without a GPU: stops at the device check, launches nothing
    assert attn(lib) in (-4, -6)
    assert attn(lib, num_nodes=FAKE) in (-4, -6)       # node counts are optional


def test_workspace_size_is_monotone_and_rejects_bad_shapes(lib):
    small = lib.tv_attention_workspace_size(1, 16, 8, 8, 64)
    big = lib.tv_attention_workspace_size(16, 64, 32, 8, 128)
    assert 0 < small < big
    assert lib.tv_attention_workspace_size(1, 16, 8, 8, 80) == 0
    assert lib.tv_argmax_workspace_size(16, 64, 128256) >= 16 * 64 * 8
    assert lib.tv_argmax_workspace_size(1, 0, 10) == 0


def test_accept_and_compact_argument_checks(lib):
    acc = lambda **kw: lib.tree_argmax_accept(*{**dict(l=FAKE, d=FAKE, p=FAKE, nn=NULL, B=2,
                                                        N=4, V=100,
                                                        a=FAKE, al=FAKE, ai=FAKE, b=FAKE,
                                                        ws=FAKE, wsb=1 << 30), **kw}.values(),
                                              STREAM)
    assert acc(B=0) == 0
    assert acc(l=NULL) == -1
    assert acc(N=300) == -2 and acc(V=0) == -2
    assert acc(wsb=8) == -4
    assert acc(l=ctypes.c_void_p(0x10002)) == -3
    noalloc = lambda **kw: lib.tree_argmax_accept_noalloc(
        *{**dict(l=FAKE, d=FAKE, p=FAKE, nn=NULL, B=2, N=4, V=100, a=FAKE, al=FAKE, ai=FAKE,
                 b=FAKE), **kw}.values(), STREAM)
    assert noalloc(B=0) == 0
    assert noalloc(l=NULL) == -1 and noalloc(b=NULL) == -1
    assert noalloc(N=300) == -2 and noalloc(V=0) == -2
    assert noalloc(l=ctypes.c_void_p(0x10002)) == -3
    # the static scratch holds 4 MiB of segment keys: 524256 node rows at most
    assert lib.tv_argmax_workspace_size(2047, 256, 128256) <= 4 << 20 < \
        lib.tv_argmax_workspace_size(2048, 256, 128256)
    assert noalloc(B=2048, N=256, V=128256) == -7
    assert noalloc(B=2047, N=256, V=128256) in (-6, -5)   # fits; no gfx950 here
    cmp_ = lambda **kw: lib.kv_compact_accepted(*{**dict(kt=FAKE, vt=FAKE, kc=FAKE, vc=FAKE,
                                                          pt=FAKE, kl=FAKE, ai=FAKE, al=FAKE,
                                                          B=2, N=4, Hkv=8, D=128, P=16, mp=4,
                                                          np_=8), **kw}.values(), STREAM)
    assert cmp_(B=0) == 0
    assert cmp_(kc=NULL) == -1
    assert cmp_(P=3) == -2
    assert cmp_(Hkv=1, D=6) == -2
    assert cmp_(kt=ctypes.c_void_p(0x10004)) == -3


def tb(lib, **kw):
    a = dict(logits=FAKE, root=FAKE, table=FAKE, hot_vocab=FAKE, hot_index=FAKE, B=2, S=4, V=1000,
             H=100, k=4, budget=32, parent=FAKE, token=FAKE, joint=FAKE, num_nodes=FAKE, ws=FAKE,
             ws_bytes=1 << 40)
    a.update(kw)
    return lib.tree_build(*a.values(), STREAM)


def test_tree_build_argument_checks(lib):
    assert tb(lib, B=0) == 0
    assert tb(lib, logits=NULL) == -1 and tb(lib, num_nodes=NULL) == -1
    assert tb(lib, table=NULL) == -1                      # hot tokens need their table
    assert tb(lib, S=0) == -2 and tb(lib, S=17) == -2
    assert tb(lib, k=0) == -2 and tb(lib, k=17) == -2 and tb(lib, k=5, V=4, H=0) == -2
    assert tb(lib, H=1001) == -2 and tb(lib, H=-1) == -2
    assert tb(lib, budget=0) == -2 and tb(lib, budget=257) == -2
    assert tb(lib, logits=ctypes.c_void_p(0x10002)) == -3
    assert tb(lib, ws=ctypes.c_void_p(0x10004)) == -3
    need = lib.tv_tree_build_workspace_size(2, 4, 1000, 100, 4)
    assert need > 0 and tb(lib, ws_bytes=need - 1) == -4
    assert lib.tv_tree_build_workspace_size(2, 0, 1000, 100, 4) == 0


def test_tree_resample_argument_checks(lib):
    def rs(**kw):
        a = dict(logits=FAKE, bonus=FAKE, alen=FAKE, table=FAKE, hot_vocab=FAKE, hot_index=FAKE,
                 B=2, S=4, V=1000, H=100, k=4, r=1, budget=32, parent=FAKE, token=FAKE,
                 joint=FAKE, num_nodes=FAKE, ws=FAKE, ws_bytes=1 << 40)
        a.update(kw)
        return lib.tree_resample(*a.values(), STREAM)
    assert rs(B=0) == 0
    assert rs(bonus=NULL) == -1 and rs(alen=NULL) == -1
    assert rs(r=-1) == -2 and rs(S=17) == -2 and rs(budget=0) == -2
    assert rs(ws_bytes=lib.tv_tree_build_workspace_size(2, 4, 1000, 100, 4) - 1) == -4



def test_lm_head_argument_checks(lib):
    def lm(**kw):
        a = dict(hidden=FAKE, w=FAKE, draft=FAKE, parent=FAKE, num_nodes=NULL, B=2, N=64,
                 V=1000, d=256, amax=FAKE, alen=FAKE, aidx=FAKE, bonus=FAKE, ws=FAKE,
                 ws_bytes=1 << 40)
        a.update(kw)
        return lib.tree_lm_head_argmax_accept(*a.values(), STREAM)
    assert lm(B=0) == 0
    assert lm(hidden=NULL) == -1 and lm(w=NULL) == -1 and lm(bonus=NULL) == -1
    assert lm(ws=NULL) == -1
    assert lm(d=0) == -2 and lm(d=48) == -2 and lm(d=32) == -2 and lm(d=96) == -2   # d: multiple of 64
    assert lm(V=0) == -2 and lm(N=257) == -2 and lm(B=65536) == -2
    assert lm(B=65535, N=256, V=(1 << 31) - 257) == -2                  # grid above 2^31 - 1
    assert lm(B=1, N=1, V=(1 << 31) - 256) == -2                        # tile ids past 2^31 - 1
    assert lm(hidden=ctypes.c_void_p(0x10008)) == -3 and lm(w=ctypes.c_void_p(0x10008)) == -3
    assert lm(ws=ctypes.c_void_p(0x10004)) == -3
    need = lib.tv_lm_head_workspace_size(2, 64, 1000, 256)
    assert need >= 2 * 64 * 8 and lm(ws_bytes=need - 1) == -4
    assert lib.tv_lm_head_workspace_size(2, 64, 1000, 40) == 0
