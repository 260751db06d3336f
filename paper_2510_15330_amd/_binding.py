"""ctypes binding of libbellman.so: argument marshalling only."""
from __future__ import annotations

import ctypes
import math
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# BELLMAN_LIBRARY selects another build of the same library (the host
# sanitizer build of paper_2510_15330_amd/build.py --sanitize)
_LIB_PATH = os.environ.get("BELLMAN_LIBRARY") or os.path.join(_HERE, "libbellman.so")

BF16, FP8_E4M3FN, INT32, FP32 = 1, 2, 3, 4
MAX_DIMS = 5
FIXED_SCRATCH_BYTES = 32 << 20     # BELLMAN_FIXED_SCRATCH_BYTES


class BellmanError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"libbellman error {code}: {msg}")
        self.code = code


class Tensor(ctypes.Structure):
    _fields_ = [
        ("data", ctypes.c_void_p),
        ("dtype", ctypes.c_int32),
        ("ndim", ctypes.c_int32),
        ("shape", ctypes.c_int64 * MAX_DIMS),
        ("stride", ctypes.c_int64 * MAX_DIMS),
        ("dequant_scale", ctypes.c_void_p),
    ]


class AttnOpts(ctypes.Structure):
    _fields_ = [("max_waves", ctypes.c_int32), ("xcd_skew", ctypes.c_int32),
                ("pages_per_step", ctypes.c_int32), ("pipeline_depth", ctypes.c_int32),
                ("event_begin", ctypes.c_void_p), ("event_end", ctypes.c_void_p),
                ("wave_times", ctypes.c_void_p)]


class PrefillOpts(ctypes.Structure):
    _fields_ = [("event_begin", ctypes.c_void_p), ("event_end", ctypes.c_void_p)]


CTL_LINEAR, CTL_MPC, CTL_BBR, CTL_PCC = 1, 2, 3, 4


class CtlParams(ctypes.Structure):
    _fields_ = [
        ("kind", ctypes.c_int32), ("window", ctypes.c_int32),
        ("t1", ctypes.c_double), ("t2", ctypes.c_double), ("r_min", ctypes.c_double), ("r_max", ctypes.c_double),
        ("horizon", ctypes.c_int32), ("floor_window", ctypes.c_int32), ("tau", ctypes.c_double),
        ("w_lat", ctypes.c_double), ("w_quality", ctypes.c_double), ("w_energy", ctypes.c_double),
        ("w_delta", ctypes.c_double), ("step", ctypes.c_double),
        ("bw_window", ctypes.c_int32), ("rt_window", ctypes.c_int32), ("cycle", ctypes.c_int32),
        ("reserved0", ctypes.c_int32), ("margin", ctypes.c_double), ("bbr_step", ctypes.c_double),
        ("probe", ctypes.c_double), ("interval", ctypes.c_int32), ("reserved1", ctypes.c_int32),
        ("epsilon", ctypes.c_double), ("gain", ctypes.c_double), ("pcc_w_lat", ctypes.c_double),
        ("pcc_w_quality", ctypes.c_double),
    ]


class CtlObs(ctypes.Structure):
    _fields_ = [("has_sample", ctypes.c_int32), ("reserved", ctypes.c_int32), ("tbt_avg", ctypes.c_double),
                ("tokens", ctypes.c_double), ("tick_s", ctypes.c_double)]


class ClassPolicy(ctypes.Structure):
    _fields_ = [("weight", ctypes.c_double), ("bypass_len", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class LoadSignal(ctypes.Structure):
    _fields_ = [
        ("controller", ctypes.c_void_p),
        ("has_sample", ctypes.c_int32),
        ("tbt_avg", ctypes.c_double),
        ("predicted_len", ctypes.c_int32),
    ]


_lib = None


def library_path() -> str:
    return _LIB_PATH


def library():
    """Load libbellman.so (built in-tree); raise if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError(f"{_LIB_PATH} is not built; run __graft_entry__.build() "
                           "(hipcc, gfx950) first — there is no fallback path")
    lib = ctypes.CDLL(_LIB_PATH)
    P, T = ctypes.c_void_p, ctypes.POINTER(Tensor)
    lib.bellman_kv_append.argtypes = [T, T, T, T, T, T, P]
    lib.bellman_kv_append.restype = ctypes.c_int
    lib.bellman_decode_attention.argtypes = [T, T, T, T, T, ctypes.c_float, T, P]
    lib.bellman_decode_attention.restype = ctypes.c_int
    lib.bellman_decode_attention_opts.argtypes = [T, T, T, T, T, ctypes.c_float, T,
                                                  ctypes.POINTER(AttnOpts), P]
    lib.bellman_decode_attention_opts.restype = ctypes.c_int
    lib.bellman_decode_attention_noalloc.argtypes = [T, T, T, T, T, ctypes.c_float, T,
                                                     ctypes.POINTER(AttnOpts), P]
    lib.bellman_decode_attention_noalloc.restype = ctypes.c_int
    lib.bellman_decode_step.argtypes = [T, T, T, T, T, T, T, ctypes.c_float, T, ctypes.POINTER(AttnOpts), P]
    lib.bellman_decode_step.restype = ctypes.c_int
    lib.bellman_probe_gather.argtypes = [P, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, P, P]
    lib.bellman_probe_gather.restype = ctypes.c_int
    lib.bellman_kv_write.argtypes = [T, T, T, T, T, T, T, P]
    lib.bellman_kv_write.restype = ctypes.c_int
    lib.bellman_prefill_attention.argtypes = [T, T, T, T, T, T, ctypes.c_float, T, P]
    lib.bellman_prefill_attention.restype = ctypes.c_int
    lib.bellman_prefill_attention_opts.argtypes = [T, T, T, T, T, T, ctypes.c_float, T,
                                                   ctypes.POINTER(PrefillOpts), P]
    lib.bellman_prefill_attention_opts.restype = ctypes.c_int
    lib.bellman_controller_create.argtypes = [ctypes.c_double, ctypes.c_double, ctypes.c_int32,
                                              ctypes.c_double, ctypes.c_double]
    lib.bellman_controller_create.restype = P
    lib.bellman_ctl_params_default.argtypes = [ctypes.c_int32, ctypes.c_double, ctypes.c_double,
                                               ctypes.POINTER(CtlParams)]
    lib.bellman_ctl_params_default.restype = ctypes.c_int
    lib.bellman_controller_create_ex.argtypes = [ctypes.POINTER(CtlParams)]
    lib.bellman_controller_create_ex.restype = P
    lib.bellman_controller_observe.argtypes = [P, ctypes.POINTER(CtlObs)]
    lib.bellman_controller_observe.restype = ctypes.c_double
    lib.bellman_length_cap_class.argtypes = [P, ctypes.c_int32, ctypes.POINTER(ClassPolicy)]
    lib.bellman_length_cap_class.restype = ctypes.c_int32
    lib.bellman_controller_destroy.argtypes = [P]
    lib.bellman_controller_destroy.restype = None
    lib.bellman_controller_rate.argtypes = [P]
    lib.bellman_controller_rate.restype = ctypes.c_double
    lib.bellman_length_cap.argtypes = [ctypes.POINTER(LoadSignal)]
    lib.bellman_length_cap.restype = ctypes.c_int32
    lib.bellman_calibrate_thresholds.argtypes = [P, ctypes.c_int64, ctypes.POINTER(ctypes.c_double),
                                                 ctypes.POINTER(ctypes.c_double)]
    lib.bellman_calibrate_thresholds.restype = ctypes.c_int
    lib.bellman_last_error.argtypes = []
    lib.bellman_last_error.restype = ctypes.c_char_p
    lib.bellman_reserve_workspace.argtypes = [ctypes.c_int64]
    lib.bellman_reserve_workspace.restype = ctypes.c_int
    lib.bellman_device_errors.argtypes = [P, ctypes.POINTER(ctypes.c_int32)]
    lib.bellman_device_errors.restype = ctypes.c_int
    lib.bellman_shutdown.argtypes = []
    lib.bellman_shutdown.restype = None
    lib.bellman_version.argtypes = []
    lib.bellman_version.restype = ctypes.c_char_p
    _lib = lib
    return lib


def last_error() -> str:
    return library().bellman_last_error().decode()


def version() -> str:
    return library().bellman_version().decode()


def _check(rc):
    if rc != 0:
        raise BellmanError(rc, last_error())


_DTYPES = {
    torch.bfloat16: BF16,
    torch.uint8: FP8_E4M3FN,          # fp8 codes carried as bytes
    torch.float8_e4m3fn: FP8_E4M3FN,
    torch.int32: INT32,
    torch.float32: FP32,
}


def desc(t: torch.Tensor, dequant_scale: torch.Tensor | None = None) -> Tensor:
    """Descriptor of a torch tensor (no copy)."""
    if t.dtype not in _DTYPES:
        raise TypeError(f"unsupported dtype {t.dtype}")
    if t.dim() > MAX_DIMS:
        raise ValueError("too many dims")
    d = Tensor()
    d.data = t.data_ptr() if t.numel() else None
    d.dtype = _DTYPES[t.dtype]
    d.ndim = t.dim()
    for i, (s, st) in enumerate(zip(t.shape, t.stride())):
        d.shape[i] = s
        d.stride[i] = st
    if dequant_scale is not None:
        if dequant_scale.dtype != torch.float32 or not dequant_scale.is_contiguous():
            raise TypeError("dequant scales must be contiguous float32")
        d.dequant_scale = dequant_scale.data_ptr()
    return d


def _device_tensors(*ts):
    for t in ts:
        if t is not None and not t.is_cuda:
            raise ValueError("libbellman works on device tensors only")


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def kv_append(k_new, v_new, k_pages, v_pages, block_table, seq_lens, stream=None,
              k_scale=None, v_scale=None):
    """bellman_kv_append: write one token per request, then seq_lens += 1.

    bf16 rows into fp8 pools are quantised with k_scale / v_scale (the
    pools' per-(request, KV head) dequantisation scales)."""
    _device_tensors(k_new, v_new, k_pages, v_pages, block_table, seq_lens, k_scale, v_scale)
    lib = library()
    _check(lib.bellman_kv_append(desc(k_new), desc(v_new), desc(k_pages, k_scale), desc(v_pages, v_scale),
                                 desc(block_table), desc(seq_lens), _stream(stream)))


def decode_attention(q, k_pages, v_pages, block_table, seq_lens, scale, out, stream=None,
                     k_scale=None, v_scale=None, max_waves=0, xcd_skew=0, events=None,
                     pages_per_step=0, pipeline_depth=0, wave_times=None):
    """bellman_decode_attention(_opts): one decode step over the paged cache.

    ``events`` is an optional pair of recorded-once torch.cuda.Event objects
    that the library records around its main attention kernel; ``xcd_skew``
    is 0 (the library's choice), -1 (equal shares) or 1..255; ``wave_times``
    an optional device int64 tensor of 3 entries per wave for the per-wave
    timing records."""
    _device_tensors(q, k_pages, v_pages, block_table, seq_lens, out, k_scale, v_scale, wave_times)
    lib = library()
    args = (desc(q), desc(k_pages, k_scale), desc(v_pages, v_scale), desc(block_table),
            desc(seq_lens), ctypes.c_float(scale), desc(out))
    if (max_waves == 0 and xcd_skew == 0 and events is None and pages_per_step == 0 and pipeline_depth == 0
            and wave_times is None):
        _check(lib.bellman_decode_attention(*args, _stream(stream)))
    else:
        ev0 = ev1 = None
        if events is not None:
            ev0, ev1 = events[0].cuda_event, events[1].cuda_event
            if not ev0 or not ev1:
                raise ValueError("record each event once before passing it")
        wt = None if wave_times is None else wave_times.data_ptr()
        opts = AttnOpts(int(max_waves), int(xcd_skew), int(pages_per_step), int(pipeline_depth), ev0, ev1, wt)
        _check(lib.bellman_decode_attention_opts(*args, ctypes.byref(opts), _stream(stream)))


def decode_attention_noalloc(q, k_pages, v_pages, block_table, seq_lens, scale, out, stream=None,
                             k_scale=None, v_scale=None, max_waves=0, xcd_skew=0, pages_per_step=0,
                             pipeline_depth=0):
    """bellman_decode_attention_noalloc: decode_attention with its scratch in
    the device's fixed array (no device allocation)."""
    _device_tensors(q, k_pages, v_pages, block_table, seq_lens, out, k_scale, v_scale)
    opts = AttnOpts(int(max_waves), int(xcd_skew), int(pages_per_step), int(pipeline_depth), None, None)
    _check(library().bellman_decode_attention_noalloc(
        desc(q), desc(k_pages, k_scale), desc(v_pages, v_scale), desc(block_table), desc(seq_lens),
        ctypes.c_float(scale), desc(out), ctypes.byref(opts), _stream(stream)))


def decode_step(k_new, v_new, q, k_pages, v_pages, block_table, seq_lens, scale, out, stream=None,
                k_scale=None, v_scale=None, max_waves=0, xcd_skew=0, events=None, pages_per_step=0,
                pipeline_depth=0, wave_times=None):
    """bellman_decode_step: kv_append of (k_new, v_new) and decode_attention
    of q in one call (the append fused into the attention launch)."""
    _device_tensors(k_new, v_new, q, k_pages, v_pages, block_table, seq_lens, out, k_scale, v_scale, wave_times)
    ev0 = ev1 = None
    if events is not None:
        ev0, ev1 = events[0].cuda_event, events[1].cuda_event
        if not ev0 or not ev1:
            raise ValueError("record each event once before passing it")
    wt = None if wave_times is None else wave_times.data_ptr()
    opts = AttnOpts(int(max_waves), int(xcd_skew), int(pages_per_step), int(pipeline_depth), ev0, ev1, wt)
    _check(library().bellman_decode_step(
        desc(k_new), desc(v_new), desc(q), desc(k_pages, k_scale), desc(v_pages, v_scale), desc(block_table),
        desc(seq_lens), ctypes.c_float(scale), desc(out), ctypes.byref(opts), _stream(stream)))


def probe_gather(pool, tile_bytes, sink, max_waves=0, stream=None):
    """bellman_probe_gather: read every tile of the device buffer ``pool``
    once in the decode kernels' scattered page pattern and XOR its words into
    ``sink`` (a cleared device int32/uint32 tensor of one element)."""
    _device_tensors(pool, sink)
    _check(library().bellman_probe_gather(ctypes.c_void_p(pool.data_ptr()), pool.numel() * pool.element_size(),
                                          int(tile_bytes), int(max_waves), ctypes.c_void_p(sink.data_ptr()),
                                          _stream(stream)))


def kv_write(k_new, v_new, k_pages, v_pages, block_table, seq_lens, q_start, stream=None):
    """bellman_kv_write: write each request's new prompt tokens after its
    cached ones, then seq_lens += tokens written."""
    _device_tensors(k_new, v_new, k_pages, v_pages, block_table, seq_lens, q_start)
    _check(library().bellman_kv_write(desc(k_new), desc(v_new), desc(k_pages), desc(v_pages), desc(block_table),
                                      desc(seq_lens), desc(q_start), _stream(stream)))


def prefill_attention(q, k_pages, v_pages, block_table, seq_lens, q_start, scale, out, stream=None,
                      events=None, k_scale=None, v_scale=None):
    """bellman_prefill_attention(_opts): causal attention of each request's
    new (last) tokens over its cached ones (fp8 pools with their
    per-(request, KV head) dequantisation scales k_scale / v_scale)."""
    _device_tensors(q, k_pages, v_pages, block_table, seq_lens, q_start, out, k_scale, v_scale)
    lib = library()
    args = (desc(q), desc(k_pages, k_scale), desc(v_pages, v_scale), desc(block_table), desc(seq_lens),
            desc(q_start), ctypes.c_float(scale), desc(out))
    if events is None:
        _check(lib.bellman_prefill_attention(*args, _stream(stream)))
        return
    ev0 = ev1 = None
    if events is not None:
        ev0, ev1 = events[0].cuda_event, events[1].cuda_event
        if not ev0 or not ev1:
            raise ValueError("record each event once before passing it")
    opts = PrefillOpts(ev0, ev1)
    _check(lib.bellman_prefill_attention_opts(*args, ctypes.byref(opts), _stream(stream)))


def reserve_workspace(nbytes: int):
    _check(library().bellman_reserve_workspace(int(nbytes)))


def device_errors(stream=None) -> int:
    v = ctypes.c_int32(0)
    _check(library().bellman_device_errors(_stream(stream), ctypes.byref(v)))
    return v.value


def shutdown():
    library().bellman_shutdown()


class Controller:
    """beLLMan's linear length controller (host only)."""

    def __init__(self, t1, t2, window=5, r_min=0.05, r_max=0.20):
        self._lib = library()
        self._h = self._lib.bellman_controller_create(float(t1), float(t2), int(window),
                                                      float(r_min), float(r_max))
        if not self._h:
            raise ValueError("invalid controller parameters")

    def close(self):
        if self._h:
            self._lib.bellman_controller_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def rate(self) -> float:
        return self._lib.bellman_controller_rate(self._h)

    def length_cap(self, predicted_len, tbt_avg=None):
        return length_cap(self, predicted_len, tbt_avg)


def length_cap(controller: Controller, predicted_len: int, tbt_avg: float | None = None) -> int:
    """bellman_length_cap: optionally push one per-second TBT average, then
    return the cap N for a request of predicted unbounded length L."""
    sig = LoadSignal(controller._h, 0 if tbt_avg is None else 1,
                     0.0 if tbt_avg is None else float(tbt_avg), int(predicted_len))
    n = library().bellman_length_cap(ctypes.byref(sig))
    if n < 0:
        raise BellmanError(n, "invalid load signal")
    return n


def ctl_params(kind, t1=0.0, t2=0.0, **overrides) -> CtlParams:
    """bellman_ctl_params_default for `kind`, then the given fields."""
    p = CtlParams()
    _check(library().bellman_ctl_params_default(int(kind), float(t1), float(t2), ctypes.byref(p)))
    for k, v in overrides.items():
        if k not in dict(CtlParams._fields_):
            raise TypeError(f"unknown controller parameter {k!r}")
        setattr(p, k, v)
    return p


class VariantController:
    """A controller of any kind (bellman_controller_create_ex), fed one tick
    at a time with observe()."""

    def __init__(self, kind, t1=0.0, t2=0.0, **overrides):
        self.params = ctl_params(kind, t1, t2, **overrides)
        self._h = library().bellman_controller_create_ex(ctypes.byref(self.params))
        if not self._h:
            raise BellmanError(-1, "invalid controller parameters")

    def close(self):
        if self._h:
            library().bellman_controller_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def rate(self) -> float:
        return library().bellman_controller_rate(self._h)

    def observe(self, has_sample, tbt=0.0, tokens=0.0, tick_s=1.0) -> float:
        o = CtlObs(int(bool(has_sample)), 0, float(tbt), float(tokens), float(tick_s))
        r = library().bellman_controller_observe(self._h, ctypes.byref(o))
        if r < 0:
            raise BellmanError(int(r), last_error() or "controller rejected the tick")
        return r

    def cap(self, predicted_len, weight=1.0, bypass_len=0) -> int:
        pol = ClassPolicy(float(weight), int(bypass_len), 0)
        n = library().bellman_length_cap_class(self._h, int(predicted_len), ctypes.byref(pol))
        if n < 0:
            raise BellmanError(n, "length cap rejected its arguments")
        return n


def calibrate_thresholds(tbt):
    """(T1, T2) = (median, 75th percentile) of an unbounded run's TBTs."""
    import numpy as np
    a = np.ascontiguousarray(np.asarray(tbt, dtype=np.float64))
    t1, t2 = ctypes.c_double(), ctypes.c_double()
    rc = library().bellman_calibrate_thresholds(a.ctypes.data_as(ctypes.c_void_p), a.size,
                                                ctypes.byref(t1), ctypes.byref(t2))
    if rc != 0:
        raise BellmanError(rc, "invalid TBT samples")
    return t1.value, t2.value
