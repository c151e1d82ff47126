"""The oracle's pins catch plausible mistakes (CPU only).

Each case plants one mistake in a temporary copy of the oracle (a dropped
term, a wrong sign or index, a transposed operand, an off-by-one in a walk,
the wrong tie rule, ...), runs the pin tests of the affected function against
that copy, and requires at least one pin to fail. An unplanted copy must pass
the same pins, so a failure is the mistake's and not the harness's."""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

ATT = ["tests/test_oracle_attention.py"]
ACC = ["tests/test_oracle_accept.py"]
RAG = ["tests/test_oracle_ragged.py"]
TB = ["tests/test_oracle_tree_build.py"]
LM = ["tests/test_oracle_lm_head.py"]

# (name, file under oracle/, text, replacement, pin files)
MUTATIONS = [
    # tree attention (oracle.c)
    ("node does not see itself", "oracle.c",
     "for (int j = i; j >= 0; j = parent[(long)b * N + j]) {",
     "for (int j = parent[(long)b * N + i]; j >= 0; j = parent[(long)b * N + j]) {", ATT),
    ("GQA head interleaved", "oracle.c", "const int g = h / G;", "const int g = h % Hkv;", ATT),
    ("softmax scale dropped", "oracle.c", "s[j] = scale * dot;", "s[j] = dot;", ATT),
    ("last prefix key dropped", "oracle.c", "for (int t = 0; t < L; ++t) {", "for (int t = 0; t < L - 1; ++t) {", ATT),
    ("page slot reversed", "oracle.c", "long off = ((pg * P + t % P) * Hkv + g) * D;",
     "long off = ((pg * P + (P - 1 - t % P)) * Hkv + g) * D;", ATT),
    ("exponent sign flipped", "oracle.c", "s[j] = exp(s[j] - m);", "s[j] = exp(m - s[j]);", ATT),
    ("max missing from lse", "oracle.c", "*lse_out = m + log(denom);", "*lse_out = log(denom);", ATT),
    ("values read from keys", "oracle.c", "vrow[n] = v_tree + off;", "vrow[n] = k_tree + off;", ATT),
    ("normaliser dropped", "oracle.c", "o[d] /= denom;", "o[d] /= 1.0;", ATT),
    # argmax and accept (oracle.c)
    ("argmax ties to the last index", "oracle.c", "if (x[v] > x[best])", "if (x[v] >= x[best])", ACC),
    ("accept ignores the parent", "oracle.c", "acc[i] = acc[p] && tok[i] == am[p];",
     "acc[i] = tok[i] == am[p];", ACC),
    ("accept compares the child's argmax", "oracle.c", "acc[i] = acc[p] && tok[i] == am[p];",
     "acc[i] = acc[p] && tok[i] == am[i];", ACC),
    ("deepest node ties to the last", "oracle.c", "depth[i] > depth[sel]))", "depth[i] >= depth[sel]))", ACC),
    ("bonus from the parent", "oracle.c", "bonus[b] = sel < 0 ? -1 : am[sel];",
     "bonus[b] = sel < 0 ? -1 : am[par[sel] < 0 ? sel : par[sel]];", ACC),
    ("compaction one slot late", "oracle.c", "int pos = kv_len[b] + j;", "int pos = kv_len[b] + j + 1;", ACC),
    ("compaction path reversed", "oracle.c", "int node = accept_idx[(long)b * N + j];",
     "int node = accept_idx[(long)b * N + (accept_len[b] - 1 - j)];", ACC),
    ("padding counts ignored", "oracle.c", "return num_nodes ? num_nodes[b] : N;", "return N;", RAG),
    # draft-tree builder and re-sampling (tree_build.py)
    ("token information dropped", "tree_build.py", "x[hot] = (l_i[hot] + row).astype(np.float32)",
     "x[hot] = l_i[hot]", TB),
    ("table transposed", "tree_build.py", "row = table[h]", "row = table[:, h]", TB),
    ("joint not a product", "tree_build.py", "joint.append(joint[f] * p)", "joint.append(p)", TB),
    ("frontier by own probability", "tree_build.py", "ranked = sorted(children, key=lambda n: (-joint[n], n))",
     "ranked = sorted(children, key=lambda n: (-prob[n], n))", TB),
    ("top-k ties to the higher id", "tree_build.py",
     "order = np.lexsort((np.arange(x.shape[0]), -x.astype(np.float64)))",
     "order = np.lexsort((-np.arange(x.shape[0]), -x.astype(np.float64)))", TB),
    ("softmax over hot tokens only", "tree_build.py", "s = np.exp(x64 - m).sum()",
     "s = np.exp(x64[hot] - m).sum() if hot.shape[0] else np.exp(x64 - m).sum()", TB),
    ("frontier of k + 1", "tree_build.py", "frontier = ranked[:k]", "frontier = ranked[:k + 1]", TB),
    # LM head (lm_head.py)
    ("vocabulary chunk offset", "lm_head.py", "cand_i = np.concatenate([top_i, c2 + v0], axis=1)",
     "cand_i = np.concatenate([top_i, c2 + v0 + 1], axis=1)", LM),
    ("LM-head ties to the higher id", "lm_head.py", "order = np.lexsort((cand_i, -cand_v), axis=1)[:, :2]",
     "order = np.lexsort((-cand_i, -cand_v), axis=1)[:, :2]", LM),
    ("hidden state transposed onto the weight", "lm_head.py", "lg = h @ w.T", "lg = h[:, ::-1] @ w.T", LM),
]


def _copy_tree(dst):
    for sub in ("oracle", "tests", "paper_2602_21224_amd"):
        shutil.copytree(os.path.join(ROOT, sub), os.path.join(dst, sub),
                        ignore=shutil.ignore_patterns("*.so", "*.so.*", "__pycache__", "csrc"))
    shutil.copy(os.path.join(ROOT, "pytest.ini"), dst)


def _run_pins(case):
    name, fname, old, new, pins = case
    d = tempfile.mkdtemp(prefix="oracle_mut_")
    try:
        _copy_tree(d)
        if fname is not None:
            path = os.path.join(d, "oracle", fname)
            src = open(path).read()
            if src.count(old) != 1:
                return name, "planting failed: text occurs %d times" % src.count(old)
            with open(path, "w") as fh:
                fh.write(src.replace(old, new))
        r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                            "-m", "not gpu", *pins], cwd=d, capture_output=True, text=True,
                           timeout=600)
        return name, r.returncode
    finally:
        shutil.rmtree(d, ignore_errors=True)


def test_unplanted_copy_passes_the_pins():
    pins = sorted({p for m in MUTATIONS for p in m[4]})
    name, rc = _run_pins(("unplanted", None, "", "", pins))
    assert rc == 0, f"the harness copy fails its own pins (rc {rc})"


def test_every_planted_mistake_fails_a_pin():
    with ThreadPoolExecutor(max_workers=min(6, os.cpu_count() or 1)) as pool:
        results = list(pool.map(_run_pins, MUTATIONS))
    missed = [(n, rc) for n, rc in results if rc == 0 or isinstance(rc, str)]
    assert not missed, f"mistakes no pin caught (or could not be planted): {missed}"
