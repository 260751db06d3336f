"""Build libbellman.so in-tree with hipcc for gfx950.

``python -m paper_2510_15330_amd.build --sanitize OUT.so`` builds the same
library with the host code of its C++ sources (descriptor validation,
workspace, controllers, serving model) under AddressSanitizer and
UndefinedBehaviorSanitizer, for runs of the CPU test suite (the device code
is built as usual; GPU sanitizers are not used).
"""
from __future__ import annotations

import os
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libbellman.so")
DEVICE_SOURCES = ["kernels.hip", "prefill.hip", "device_state.hip", "probe.hip"]
HOST_SOURCES = ["bellman_api.cpp", "controller.cpp", "serve_sim.cpp"]
SOURCES = DEVICE_SOURCES + HOST_SOURCES

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    "-Wall", "-Wno-unused-command-line-argument",
    # no packed FP32 instructions in generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]
# host-side sanitizers only (each flag scoped to the host compilation)
SANITIZE_FLAGS = ["-g", "-Xarch_host", "-fsanitize=address,undefined", "-Xarch_host", "-fno-sanitize-recover=all",
                  "-Xarch_host", "-fno-omit-frame-pointer"]


def hipcc():
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    path = os.path.join(rocm, "bin", "hipcc")
    return path if os.path.exists(path) else "hipcc"


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in res.stdout.splitlines() if "packed-fp32-ops" not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{out}")
    if verbose and out.strip():
        print(out)


def _build(out: str, sanitize: bool, verbose: bool) -> str:
    """Compile the sources in parallel, then link them into `out`."""
    from concurrent.futures import ThreadPoolExecutor
    with tempfile.TemporaryDirectory() as d:
        objs = [os.path.join(d, src + ".o") for src in SOURCES]

        def compile_one(i):
            src = SOURCES[i]
            flags = HIPCC_FLAGS + (SANITIZE_FLAGS if sanitize and src in HOST_SOURCES else [])
            _run([hipcc()] + flags + ["-c", os.path.join(CSRC, src), "-o", objs[i]], verbose)

        with ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
            list(ex.map(compile_one, range(len(SOURCES))))
        link = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC"]
        if sanitize:
            link += ["-Xarch_host", "-fsanitize=address,undefined", "-shared-libsan"]
        _run(link + objs + ["-o", out], verbose)
    return out


def build(verbose: bool = False) -> str:
    tmp = LIB + f".tmp{os.getpid()}"
    _build(tmp, False, verbose)
    os.replace(tmp, LIB)
    return LIB


def build_sanitized(out: str, verbose: bool = False) -> str:
    """The library with its C++ host sources under ASan + UBSan, at `out`."""
    return _build(out, True, verbose)


if __name__ == "__main__":
    if "--sanitize" in sys.argv:
        i = sys.argv.index("--sanitize")
        print(build_sanitized(sys.argv[i + 1], verbose="-v" in sys.argv))
    else:
        build(verbose="-v" in sys.argv)
        print(LIB)
