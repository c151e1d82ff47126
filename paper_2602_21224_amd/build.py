"""Build libtreeverify.so (gfx950 only) in-tree with hipcc."""
from __future__ import annotations

import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libtreeverify.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    "-fvisibility=hidden", "-munsafe-fp-atomics",
    # keep the compiler from emitting packed fp32 VALU ops
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
]
_NOISE = "is not a recognized feature for this target"


def sources():
    return sorted(glob.glob(os.path.join(HERE, "csrc", "*.hip")))


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in (r.stderr or "").splitlines() if _NOISE not in l)
    return r.returncode, err


def build(verbose: bool = False, extra_flags=(), out: str = LIB) -> str:
    """Compile every source to an object in parallel, then link the shared
    library; the result replaces `out` only when every step succeeded."""
    import shutil
    import tempfile
    from concurrent.futures import ThreadPoolExecutor
    tmpdir = tempfile.mkdtemp(prefix="treeverify_build_")
    objs = [os.path.join(tmpdir, os.path.basename(src)[:-4] + ".o") for src in sources()]
    cmds = [[HIPCC, *FLAGS, *extra_flags, "-c", src, "-o", obj]
            for src, obj in zip(sources(), objs)]
    try:
        with ThreadPoolExecutor(max_workers=min(len(cmds), os.cpu_count() or 1)) as pool:
            results = list(pool.map(_run, cmds))
        for cmd, (rc, err) in zip(cmds, results):
            if verbose:
                print(" ".join(cmd), flush=True)
            if rc != 0:
                raise RuntimeError(f"hipcc failed on {cmd[-3]}:\n" + err)
            if verbose and err.strip():
                print(err, file=sys.stderr)
        tmp = os.path.join(tmpdir, "lib.so")
        rc, err = _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp])
        if rc != 0:
            raise RuntimeError("link failed:\n" + err)
        shutil.copyfile(tmp, out + ".part")
        os.chmod(out + ".part", 0o755)
        os.replace(out + ".part", out)
    finally:
        shutil.rmtree(tmpdir, ignore_errors=True)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
