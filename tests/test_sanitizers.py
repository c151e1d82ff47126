"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

* The oracle (plain C) is built with gcc's ASan + UBSan and its pin tests run
  against that build.
* The library is built with its host code (argument checks, launch
  arithmetic, workspace carving) under clang's ASan + UBSan, device code as
  usual, and the host-side ABI checks run against that build.
Any sanitizer report fails the run (no recovery from UB, leak checking off:
the interpreter itself is not instrumented)."""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
def _san_env(logdir):
    """Sanitizer options: no recovery, leak checking off, reports to files."""
    return {"ASAN_OPTIONS": f"detect_leaks=0:abort_on_error=1:log_path={logdir}/asan",
            "UBSAN_OPTIONS": f"print_stacktrace=1:halt_on_error=1:log_path={logdir}/ubsan"}


def _run(cmd, env, cwd=ROOT):
    e = dict(os.environ)
    e.update(env)
    return subprocess.run(cmd, cwd=cwd, env=e, capture_output=True, text=True, timeout=900)


def _assert_clean(r, logdir, what):
    reports = [os.path.join(logdir, f) for f in os.listdir(logdir)
               if f.startswith("asan") or f.startswith("ubsan")]
    text = "".join(open(f).read() for f in reports)
    assert not reports, f"{what}: sanitizer reports:\n{text[-4000:]}"
    out = r.stdout + r.stderr
    assert r.returncode == 0, f"{what} failed (rc {r.returncode}):\n{out[-4000:]}"


def test_oracle_pins_under_asan_and_ubsan():
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not available")
    libasan = subprocess.run([gcc, "-print-file-name=libasan.so"], capture_output=True,
                             text=True).stdout.strip()
    libubsan = subprocess.run([gcc, "-print-file-name=libubsan.so"], capture_output=True,
                              text=True).stdout.strip()
    d = tempfile.mkdtemp(prefix="oracle_san_")
    try:
        lib = os.path.join(d, "liboracle_san.so")
        subprocess.run([gcc, "-O1", "-g", "-std=c11", "-fopenmp", "-ffp-contract=off",
                        "-fno-fast-math", "-fsanitize=address,undefined",
                        "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-shared", "-fPIC",
                        os.path.join(ROOT, "oracle", "oracle.c"), "-o", lib, "-lm"], check=True)
        r = _run([sys.executable, "-m", "pytest", "-q", "-s", "-x", "-p", "no:cacheprovider",
                  "-m", "not gpu", "tests/test_oracle_attention.py", "tests/test_oracle_accept.py",
                  "tests/test_oracle_ragged.py"],
                 {**_san_env(d), "TREEVERIFY_ORACLE_LIB": lib, "LD_PRELOAD": f"{libasan}:{libubsan}"})
        _assert_clean(r, d, "oracle pins under ASan/UBSan")
    finally:
        shutil.rmtree(d, ignore_errors=True)


def test_library_host_checks_under_asan_and_ubsan():
    from paper_2602_21224_amd import build
    if not os.path.exists(build.HIPCC):
        pytest.skip("hipcc not available")
    rt = subprocess.run([build.HIPCC, "-print-file-name=libclang_rt.asan-x86_64.so"],
                        capture_output=True, text=True).stdout.strip()
    if not os.path.isabs(rt) or not os.path.exists(rt):
        import glob
        cands = glob.glob("/opt/rocm/lib/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
        if not cands:
            pytest.skip("clang's ASan runtime not found")
        rt = cands[0]
    d = tempfile.mkdtemp(prefix="lib_san_")
    try:
        lib = os.path.join(d, "libtreeverify_san.so")
        host = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer",
                "-Xarch_host", "-g"]
        build.build(extra_flags=host, out=lib)
        r = _run([sys.executable, "-m", "pytest", "-q", "-s", "-x", "-p", "no:cacheprovider",
                  "tests/test_abi.py"],
                 {**_san_env(d), "TREEVERIFY_LIB": lib, "LD_PRELOAD": rt})
        _assert_clean(r, d, "host ABI checks under ASan/UBSan")
    finally:
        shutil.rmtree(d, ignore_errors=True)
