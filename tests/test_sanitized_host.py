"""The host code under AddressSanitizer and UndefinedBehaviorSanitizer: the
library's C++ sources (descriptor validation, workspace bookkeeping,
controllers, serving model) and the oracle are rebuilt with the sanitizers
(paper_2510_15330_amd/build.py --sanitize, oracle.build_sanitized) and the CPU
tests that drive native code run against those builds in a child process,
which aborts on the first report.  No GPU is used (GPU sanitizers are not)."""
from __future__ import annotations

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
NATIVE_TESTS = ["tests/test_abi.py", "tests/test_controller_lib.py", "tests/test_controller_variants_lib.py",
                "tests/test_serve_sim.py", "tests/test_oracle_pins.py", "tests/test_oracle_prefill.py",
                "tests/test_oracle_quant.py"]

pytestmark = pytest.mark.skipif(os.environ.get("BELLMAN_SANITIZED_RUN") == "1", reason="inside the sanitized run")


def _asan_runtime():
    clang = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "llvm", "bin", "clang")
    return subprocess.check_output([clang, "-print-file-name=libclang_rt.asan-x86_64.so"], text=True).strip()


def test_native_tests_clean_under_asan_and_ubsan(tmp_path):
    sys.path.insert(0, ROOT)
    import oracle
    from paper_2510_15330_amd import build as B
    lib = B.build_sanitized(str(tmp_path / "libbellman_san.so"))
    olib = oracle.build_sanitized(str(tmp_path / "liboracle_san.so"))
    rt = _asan_runtime()
    assert os.path.exists(rt), rt
    env = dict(os.environ, LD_PRELOAD=rt, BELLMAN_LIBRARY=lib, ORACLE_LIBRARY=olib, BELLMAN_SANITIZED_RUN="1",
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    # the child really loads the sanitized builds
    probe = ("import paper_2510_15330_amd as bl, oracle; bl.library(); oracle.load(); "
             "m = open('/proc/self/maps').read(); "
             f"assert {lib!r} in m and {olib!r} in m and 'libclang_rt.asan' in m; print('loaded')")
    r = subprocess.run([sys.executable, "-c", probe], cwd=ROOT, env=env, capture_output=True, text=True)
    assert r.returncode == 0 and "loaded" in r.stdout, r.stdout[-2000:] + r.stderr[-2000:]
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-m", "not gpu", "-p", "no:cacheprovider"]
                       + NATIVE_TESTS, cwd=ROOT, env=env, capture_output=True, text=True)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
    assert " passed" in out
