"""Reference oracle for the decode-attention library.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this package.  It shares no code with
the GPU library (``paper_2510_15330_amd``) and never imports it.

* ``oracle.c`` — binary64 paged decode and prompt (prefill) attention, the
  byte-exact KV append and prompt write, built by gcc into ``liboracle.so``
  and called through ctypes.
* ``controller.py`` — the paper's linear length controller (Sec. 3,
  "Placeholder for congestion control", "beLLMan in action"), in plain Python.
* ``serve_sim.py`` — the closed-loop serving model (Sec. 4), an event loop in
  plain Python.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

from .controller import OracleController, calibrate_thresholds  # noqa: F401

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

BF16 = 1
FP8_E4M3FN = 2

_lib = None


def build(force: bool = True) -> str:
    """Compile ``oracle.c`` with gcc (-O2, OpenMP, no intrinsics)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.check_call(
            ["gcc", "-O2", "-fopenmp", "-std=c99", "-Wall", "-shared", "-fPIC",
             _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def build_sanitized(out: str) -> str:
    """``oracle.c`` under AddressSanitizer and UndefinedBehaviorSanitizer, at
    `out` (ROCm's clang, so that one sanitizer runtime serves it and the
    library's host build)."""
    clang = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "llvm", "bin", "clang")
    subprocess.check_call(
        [clang, "-O1", "-g", "-fopenmp", "-std=c99", "-Wall", "-shared", "-fPIC", "-fsanitize=address,undefined",
         "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-shared-libsan", _SRC, "-o", out, "-lm"])
    return out


def load(path: str | None = None):
    """Load the oracle library, building it only if no build exists."""
    global _lib
    if path is not None:
        return _bind(ctypes.CDLL(path))
    if _lib is None and os.environ.get("ORACLE_LIBRARY"):
        # another build of oracle.c (the host sanitizer build)
        _lib = _bind(ctypes.CDLL(os.environ["ORACLE_LIBRARY"]))
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        _lib = _bind(ctypes.CDLL(_LIB))
    return _lib


def _bind(lib):
    P = ctypes.c_void_p
    i32, i64 = ctypes.c_int, ctypes.c_int64
    lib.oracle_bf16_to_f64.argtypes = [ctypes.c_uint16]
    lib.oracle_bf16_to_f64.restype = ctypes.c_double
    lib.oracle_e4m3fn_to_f64.argtypes = [ctypes.c_uint8]
    lib.oracle_e4m3fn_to_f64.restype = ctypes.c_double
    lib.oracle_decode_attention.argtypes = [
        i32, i32, i32, i32, i32, P, P, P, i64, P, P, P, i32, P, ctypes.c_float, P]
    lib.oracle_decode_attention.restype = i32
    lib.oracle_kv_append.argtypes = [i32, i32, i32, i32, i32, P, P, P, P, i64, P, P, P, i32, P]
    lib.oracle_kv_append.restype = i32
    lib.oracle_prefill_attention.argtypes = [
        i32, i32, i32, i32, i32, P, P, P, i64, P, P, P, i32, P, P, ctypes.c_float, P]
    lib.oracle_prefill_attention.restype = i32
    lib.oracle_kv_write.argtypes = [i32, i32, i32, i32, P, P, P, P, i64, P, i32, P, P]
    lib.oracle_kv_write.restype = i32
    lib.oracle_quantize_e4m3fn.argtypes = [ctypes.c_float, ctypes.c_float]
    lib.oracle_quantize_e4m3fn.restype = ctypes.c_uint8
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = i32
    return lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    a = np.ascontiguousarray(a)
    assert a.dtype == dtype, (a.dtype, dtype)
    return a


def num_threads(lib=None) -> int:
    return (lib or load()).oracle_num_threads()


def bf16_to_f64(bits: int, lib=None) -> float:
    return (lib or load()).oracle_bf16_to_f64(int(bits))


def e4m3fn_to_f64(code: int, lib=None) -> float:
    return (lib or load()).oracle_e4m3fn_to_f64(int(code))


def decode_attention(q_bits, k_pages, v_pages, block_table, seq_lens, scale,
                     kv_dtype=BF16, k_scale=None, v_scale=None, lib=None):
    """Binary64 decode attention over the paged layout.

    q_bits      uint16 [B, H_q, D]   (bf16 bit patterns)
    k_pages     uint16|uint8 [NP, H_kv, D/x, 16, x]
    v_pages     uint16|uint8 [NP, H_kv, D, 16]
    block_table int32 [B, maxP];  seq_lens int32 [B] (attention lengths)
    Returns float64 [B, H_q, D].
    """
    lib = lib or load()
    q_bits = _c(q_bits, np.uint16)
    code = np.uint16 if kv_dtype == BF16 else np.uint8
    k_pages = _c(k_pages, code)
    v_pages = _c(v_pages, code)
    block_table = _c(block_table, np.int32)
    seq_lens = _c(seq_lens, np.int32)
    B, H_q, D = q_bits.shape
    NP, H_kv = k_pages.shape[0], k_pages.shape[1]
    if kv_dtype == FP8_E4M3FN:
        k_scale = _c(k_scale, np.float32)
        v_scale = _c(v_scale, np.float32)
    out = np.empty((B, H_q, D), dtype=np.float64)
    rc = lib.oracle_decode_attention(
        B, H_q, H_kv, D, kv_dtype, _ptr(q_bits), _ptr(k_pages), _ptr(v_pages), NP,
        _ptr(k_scale), _ptr(v_scale), _ptr(block_table), block_table.shape[1],
        _ptr(seq_lens), float(scale), _ptr(out))
    if rc != 0:
        raise ValueError(f"oracle_decode_attention failed: {rc}")
    return out


def quantize_e4m3fn(x: float, scale: float, lib=None) -> int:
    return (lib or load()).oracle_quantize_e4m3fn(float(x), float(scale))


def kv_append(k_new, v_new, k_pages, v_pages, block_table, seq_lens,
              kv_dtype=BF16, k_scale=None, v_scale=None, lib=None):
    """Append on host copies; mutates k_pages, v_pages, seq_lens.

    Rows of the pool's element type are copied byte for byte; bf16 rows
    (uint16 bit patterns) into fp8 pools are quantised with the per-(request,
    KV head) scales k_scale / v_scale (float32 [B, H_kv])."""
    lib = lib or load()
    code = np.uint16 if kv_dtype == BF16 else np.uint8
    for a in (k_pages, v_pages, seq_lens):
        assert a.flags.c_contiguous
    new_dtype = BF16 if np.asarray(k_new).dtype == np.uint16 else FP8_E4M3FN
    ncode = np.uint16 if new_dtype == BF16 else np.uint8
    k_new = _c(k_new, ncode)
    v_new = _c(v_new, ncode)
    assert k_pages.dtype == code and v_pages.dtype == code
    assert seq_lens.dtype == np.int32
    if new_dtype != kv_dtype:
        assert kv_dtype == FP8_E4M3FN and new_dtype == BF16
        k_scale = _c(k_scale, np.float32)
        v_scale = _c(v_scale, np.float32)
    block_table = _c(block_table, np.int32)
    B, H_kv, D = k_new.shape
    rc = lib.oracle_kv_append(B, H_kv, D, kv_dtype, new_dtype, _ptr(k_new), _ptr(v_new),
                              _ptr(k_pages), _ptr(v_pages), k_pages.shape[0],
                              _ptr(k_scale), _ptr(v_scale),
                              _ptr(block_table), block_table.shape[1], _ptr(seq_lens))
    if rc != 0:
        raise ValueError(f"oracle_kv_append failed: {rc}")


def prefill_attention(q_bits, k_pages, v_pages, block_table, seq_lens, q_start, scale,
                      kv_dtype=BF16, k_scale=None, v_scale=None, lib=None):
    """Binary64 causal prompt attention over the paged layout.

    q_bits   uint16 [T, H_q, D]; q_start int32 [B + 1] (q_start[0] = 0,
    q_start[B] = T): request b's query tokens are the last
    n_b = q_start[b+1] - q_start[b] of its seq_lens[b] cached tokens, and
    each attends every cached token up to its own position.
    Returns float64 [T, H_q, D].
    """
    lib = lib or load()
    q_bits = _c(q_bits, np.uint16)
    code = np.uint16 if kv_dtype == BF16 else np.uint8
    k_pages = _c(k_pages, code)
    v_pages = _c(v_pages, code)
    block_table = _c(block_table, np.int32)
    seq_lens = _c(seq_lens, np.int32)
    q_start = _c(q_start, np.int32)
    T, H_q, D = q_bits.shape
    B = len(seq_lens)
    NP, H_kv = k_pages.shape[0], k_pages.shape[1]
    if kv_dtype == FP8_E4M3FN:
        k_scale = _c(k_scale, np.float32)
        v_scale = _c(v_scale, np.float32)
    out = np.empty((T, H_q, D), dtype=np.float64)
    rc = lib.oracle_prefill_attention(
        B, H_q, H_kv, D, kv_dtype, _ptr(q_bits), _ptr(k_pages), _ptr(v_pages), NP,
        _ptr(k_scale), _ptr(v_scale), _ptr(block_table), block_table.shape[1],
        _ptr(seq_lens), _ptr(q_start), float(scale), _ptr(out))
    if rc != 0:
        raise ValueError(f"oracle_prefill_attention failed: {rc}")
    return out


def kv_write(k_new, v_new, k_pages, v_pages, block_table, seq_lens, q_start, kv_dtype=BF16, lib=None):
    """Prompt write on host copies; mutates k_pages, v_pages, seq_lens.
    k_new / v_new [T, H_kv, D] in the pools' element type (uint16 / uint8)."""
    lib = lib or load()
    code = np.uint16 if kv_dtype == BF16 else np.uint8
    for a in (k_pages, v_pages, seq_lens):
        assert a.flags.c_contiguous
    k_new = _c(k_new, code)
    v_new = _c(v_new, code)
    assert k_pages.dtype == code and v_pages.dtype == code and seq_lens.dtype == np.int32
    block_table = _c(block_table, np.int32)
    q_start = _c(q_start, np.int32)
    T, H_kv, D = k_new.shape
    rc = lib.oracle_kv_write(len(seq_lens), H_kv, D, kv_dtype, _ptr(k_new), _ptr(v_new), _ptr(k_pages),
                             _ptr(v_pages), k_pages.shape[0], _ptr(block_table), block_table.shape[1],
                             _ptr(seq_lens), _ptr(q_start))
    if rc != 0:
        raise ValueError(f"oracle_kv_write failed: {rc}")
