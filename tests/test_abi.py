"""Host-side checks of the C ABI: the library loads, exports every symbol the
header declares, and rejects malformed descriptors before any HIP call (so
these run without a GPU)."""
from __future__ import annotations

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bellman.h")


@pytest.fixture(scope="module")
def B():
    from paper_2510_15330_amd import _binding
    return _binding


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(bellman_[a-z0-9_]+)\s*\(", src)))


def test_exports_every_declared_symbol(B):
    lib = B.library()
    names = declared_functions()
    assert len(names) >= 12
    for n in names:
        assert hasattr(lib, n), n


FAKE = 1 << 20   # an aligned address that is never dereferenced: calls fail validation first


def t(dtype, shape, stride=None, data=FAKE, scale=None):
    d = ctypes.pointer(__import__("paper_2510_15330_amd._binding", fromlist=["Tensor"]).Tensor())
    d.contents.data = data
    d.contents.dtype = dtype
    d.contents.ndim = len(shape)
    if stride is None:
        stride, acc = [], 1
        for s in reversed(shape):
            stride.insert(0, acc)
            acc *= s
    for i, (s, st) in enumerate(zip(shape, stride)):
        d.contents.shape[i] = s
        d.contents.stride[i] = st
    d.contents.dequant_scale = scale
    return d


def good(B_, kv=1, D=128, Hq=32, Hkv=8, NP=100, Bsz=4, maxP=10):
    x = 8 if kv == B_.BF16 else 16
    sc = FAKE if kv == B_.FP8_E4M3FN else None
    return dict(
        q=t(B_.BF16, [Bsz, Hq, D]),
        k=t(kv, [NP, Hkv, D // x, 16, x], scale=sc),
        v=t(kv, [NP, Hkv, D, 16], scale=sc),
        bt=t(B_.INT32, [Bsz, maxP]),
        sl=t(B_.INT32, [Bsz]),
        out=t(B_.BF16, [Bsz, Hq, D]),
        kn=t(kv, [Bsz, Hkv, D]),
        vn=t(kv, [Bsz, Hkv, D]),
    )


def attn(B_, g, scale=0.125):
    lib = B_.library()
    return lib.bellman_decode_attention(g["q"], g["k"], g["v"], g["bt"], g["sl"], scale, g["out"], None)


def append(B_, g):
    lib = B_.library()
    return lib.bellman_kv_append(g["kn"], g["vn"], g["k"], g["v"], g["bt"], g["sl"], None)


ERR_INVALID, ERR_UNSUPPORTED = -1, -2

ATTN_CASES = [
    ("null q", lambda B_, g: g.update(q=None), ERR_INVALID, "q: null descriptor"),
    ("q wrong dtype", lambda B_, g: g.update(q=t(B_.FP32, [4, 32, 128])), ERR_INVALID, "q: dtype"),
    ("q null data", lambda B_, g: g.update(q=t(B_.BF16, [4, 32, 128], data=None)), ERR_INVALID, "null data"),
    ("head_dim 96", lambda B_, g: g.update(k=t(B_.BF16, [100, 8, 12, 16, 8]), v=t(B_.BF16, [100, 8, 96, 16]),
                                            q=t(B_.BF16, [4, 32, 96]), out=t(B_.BF16, [4, 32, 96])),
     ERR_UNSUPPORTED, "head_dim 96"),
    ("page size 32", lambda B_, g: g.update(k=t(B_.BF16, [100, 8, 16, 32, 8])), ERR_UNSUPPORTED, "page size"),
    ("H_q not multiple", lambda B_, g: g.update(q=t(B_.BF16, [4, 30, 128]), out=t(B_.BF16, [4, 30, 128])),
     ERR_INVALID, "not a multiple"),
    ("group > 16", lambda B_, g: g.update(q=t(B_.BF16, [4, 256, 128]), out=t(B_.BF16, [4, 256, 128])),
     ERR_UNSUPPORTED, "group"),
    ("non-finite scale", lambda B_, g: None, ERR_INVALID, "scale"),
    ("v shape mismatch", lambda B_, g: g.update(v=t(B_.BF16, [100, 8, 64, 16])), ERR_INVALID, "v_pages"),
    ("k/v dtype mismatch", lambda B_, g: g.update(v=t(B_.FP8_E4M3FN, [100, 8, 128, 16])), ERR_INVALID, "differs"),
    ("non-contiguous pool", lambda B_, g: g.update(k=t(B_.BF16, [100, 8, 16, 16, 8], [16384 * 2, 2048, 128, 8, 1])),
     ERR_UNSUPPORTED, "contiguous"),
    ("batch too large", lambda B_, g: g.update(q=t(B_.BF16, [9000, 32, 128]), out=t(B_.BF16, [9000, 32, 128]),
                                               bt=t(B_.INT32, [9000, 10]), sl=t(B_.INT32, [9000])),
     ERR_UNSUPPORTED, "batch 9000"),
    ("block table rows", lambda B_, g: g.update(bt=t(B_.INT32, [3, 10])), ERR_INVALID, "block_table"),
    ("block table dtype", lambda B_, g: g.update(bt=t(B_.FP32, [4, 10])), ERR_INVALID, "block_table: dtype"),
    ("seq_lens size", lambda B_, g: g.update(sl=t(B_.INT32, [5])), ERR_INVALID, "seq_lens"),
    ("out shape", lambda B_, g: g.update(out=t(B_.BF16, [4, 32, 64])), ERR_INVALID, "out: shape"),
    ("q strided inner", lambda B_, g: g.update(q=t(B_.BF16, [4, 32, 128], [8192, 256, 2])), ERR_UNSUPPORTED, "innermost"),
    ("misaligned q", lambda B_, g: g.update(q=t(B_.BF16, [4, 32, 128], data=FAKE + 2)), ERR_UNSUPPORTED, "aligned"),
    ("fp8 without scales", lambda B_, g: g.update(k=t(B_.FP8_E4M3FN, [100, 8, 8, 16, 16]),
                                                  v=t(B_.FP8_E4M3FN, [100, 8, 128, 16])), ERR_INVALID, "dequant_scale"),
    ("bf16 with scales", lambda B_, g: g.update(k=t(B_.BF16, [100, 8, 16, 16, 8], scale=FAKE)), ERR_INVALID, "dequant_scale"),
    ("empty pool", lambda B_, g: g.update(k=t(B_.BF16, [0, 8, 16, 16, 8]), v=t(B_.BF16, [0, 8, 128, 16])),
     ERR_INVALID, "no pages"),
    ("fp8 wrong chunk", lambda B_, g: g.update(k=t(B_.FP8_E4M3FN, [100, 8, 16, 16, 8], scale=FAKE),
                                               v=t(B_.FP8_E4M3FN, [100, 8, 128, 16], scale=FAKE)), ERR_INVALID, "chunk"),
]


@pytest.mark.parametrize("name,mut,code,msg", ATTN_CASES, ids=[c[0] for c in ATTN_CASES])
def test_attention_rejects(B, name, mut, code, msg):
    g = good(B)
    mut(B, g)
    rc = attn(B, g, float("nan") if name == "non-finite scale" else 0.125)
    assert rc == code
    assert msg in B.last_error()


APPEND_CASES = [
    ("k_new dtype", lambda B_, g: g.update(kn=t(B_.FP8_E4M3FN, [4, 8, 128])), ERR_INVALID, "k_new: dtype"),
    ("k_new heads", lambda B_, g: g.update(kn=t(B_.BF16, [4, 4, 128])), ERR_INVALID, "k_new: shape"),
    ("v_new batch", lambda B_, g: g.update(vn=t(B_.BF16, [3, 8, 128])), ERR_INVALID, "v_new: shape"),
    ("seq_lens null", lambda B_, g: g.update(sl=t(B_.INT32, [4], data=None)), ERR_INVALID, "null data"),
    ("misaligned k_new", lambda B_, g: g.update(kn=t(B_.BF16, [4, 8, 128], data=FAKE + 4)), ERR_UNSUPPORTED, "aligned"),
    ("misaligned v_new", lambda B_, g: g.update(vn=t(B_.BF16, [4, 8, 128], data=FAKE + 2)), ERR_UNSUPPORTED, "aligned"),
    ("quantising without scales", lambda B_, g: g.update(k=t(B_.FP8_E4M3FN, [100, 8, 8, 16, 16]),
                                                         v=t(B_.FP8_E4M3FN, [100, 8, 128, 16])),
     ERR_INVALID, "needs dequant_scale"),
    ("fp8 rows into bf16 pools", lambda B_, g: g.update(kn=t(B_.FP8_E4M3FN, [4, 8, 128]), vn=t(B_.FP8_E4M3FN, [4, 8, 128])),
     ERR_INVALID, "k_new: dtype"),
]


@pytest.mark.parametrize("name,mut,code,msg", APPEND_CASES, ids=[c[0] for c in APPEND_CASES])
def test_append_rejects(B, name, mut, code, msg):
    g = good(B)
    mut(B, g)
    assert append(B, g) == code
    assert msg in B.last_error()


def step(B_, g):
    lib = B_.library()
    return lib.bellman_decode_step(g["kn"], g["vn"], g["q"], g["k"], g["v"], g["bt"], g["sl"], 0.125, g["out"],
                                   None, None)


STEP_CASES = [
    ("k_new null", lambda B_, g: g.update(kn=None), ERR_INVALID, "k_new and v_new"),
    ("v_new null", lambda B_, g: g.update(vn=None), ERR_INVALID, "k_new and v_new"),
    ("k_new heads", lambda B_, g: g.update(kn=t(B_.BF16, [4, 4, 128])), ERR_INVALID, "k_new: shape"),
    ("v_new dtype", lambda B_, g: g.update(vn=t(B_.FP32, [4, 8, 128])), ERR_INVALID, "v_new: dtype"),
    ("misaligned v_new", lambda B_, g: g.update(vn=t(B_.BF16, [4, 8, 128], data=FAKE + 2)), ERR_UNSUPPORTED, "aligned"),
    ("fp8 rows into bf16 pools", lambda B_, g: g.update(kn=t(B_.FP8_E4M3FN, [4, 8, 128]), vn=t(B_.FP8_E4M3FN, [4, 8, 128])),
     ERR_INVALID, "k_new: dtype"),
    ("out rows", lambda B_, g: g.update(out=t(B_.BF16, [3, 32, 128])), ERR_INVALID, "out"),
]


@pytest.mark.parametrize("name,mut,code,msg", STEP_CASES, ids=[c[0] for c in STEP_CASES])
def test_step_rejects(B, name, mut, code, msg):
    # the one-call decode step validates its rows as the append does and the
    # rest as the attention does, before any HIP call
    g = good(B)
    mut(B, g)
    assert step(B, g) == code
    assert msg in B.last_error()


def prompt(B_, g, T=40, Bsz=4):
    g.update(pq=t(B_.BF16, [T, 32, 128]), pout=t(B_.BF16, [T, 32, 128]), qs=t(B_.INT32, [Bsz + 1]),
             pkn=t(B_.BF16, [T, 8, 128]), pvn=t(B_.BF16, [T, 8, 128]))
    return g


PREFILL_CASES = [
    ("q_start size", lambda B_, g: g.update(qs=t(B_.INT32, [4])), ERR_INVALID, "q_start"),
    ("q_start dtype", lambda B_, g: g.update(qs=t(B_.FP32, [5])), ERR_INVALID, "q_start: dtype"),
    ("q_start strided", lambda B_, g: g.update(qs=t(B_.INT32, [5], [2])), ERR_UNSUPPORTED, "contiguous"),
    ("out rows", lambda B_, g: g.update(pout=t(B_.BF16, [39, 32, 128])), ERR_INVALID, "out: shape"),
    ("H_q not multiple", lambda B_, g: g.update(pq=t(B_.BF16, [40, 30, 128]), pout=t(B_.BF16, [40, 30, 128])),
     ERR_INVALID, "not a multiple"),
    ("fp8 pools without scales", lambda B_, g: g.update(k=t(B_.FP8_E4M3FN, [100, 8, 8, 16, 16]),
                                                        v=t(B_.FP8_E4M3FN, [100, 8, 128, 16])), ERR_INVALID,
     "dequant_scale"),
    ("fp8 pools wrong chunk", lambda B_, g: g.update(k=t(B_.FP8_E4M3FN, [100, 8, 16, 16, 8], scale=FAKE),
                                                     v=t(B_.FP8_E4M3FN, [100, 8, 128, 16], scale=FAKE)), ERR_INVALID,
     "chunk"),
    ("misaligned q", lambda B_, g: g.update(pq=t(B_.BF16, [40, 32, 128], data=FAKE + 2)), ERR_UNSUPPORTED, "aligned"),
    ("misaligned out", lambda B_, g: g.update(pout=t(B_.BF16, [40, 32, 128], data=FAKE + 4)), ERR_UNSUPPORTED,
     "aligned"),
    ("non-finite scale", lambda B_, g: None, ERR_INVALID, "scale"),
]


@pytest.mark.parametrize("name,mut,code,msg", PREFILL_CASES, ids=[c[0] for c in PREFILL_CASES])
def test_prefill_rejects(B, name, mut, code, msg):
    g = prompt(B, good(B))
    mut(B, g)
    lib = B.library()
    scale = float("nan") if name == "non-finite scale" else 0.125
    rc = lib.bellman_prefill_attention(g["pq"], g["k"], g["v"], g["bt"], g["sl"], g["qs"], scale, g["pout"], None)
    assert rc == code
    assert msg in B.last_error()


WRITE_CASES = [
    ("k_new heads", lambda B_, g: g.update(pkn=t(B_.BF16, [40, 4, 128])), ERR_INVALID, "k_new: shape"),
    ("v_new rows", lambda B_, g: g.update(pvn=t(B_.BF16, [39, 8, 128])), ERR_INVALID, "v_new: shape"),
    ("q_start size", lambda B_, g: g.update(qs=t(B_.INT32, [6])), ERR_INVALID, "q_start"),
    ("misaligned k_new", lambda B_, g: g.update(pkn=t(B_.BF16, [40, 8, 128], data=FAKE + 8)), ERR_UNSUPPORTED,
     "aligned"),
    ("misaligned v_new", lambda B_, g: g.update(pvn=t(B_.BF16, [40, 8, 128], data=FAKE + 8)), ERR_UNSUPPORTED,
     "aligned"),
]


@pytest.mark.parametrize("name,mut,code,msg", WRITE_CASES, ids=[c[0] for c in WRITE_CASES])
def test_prompt_write_rejects(B, name, mut, code, msg):
    g = prompt(B, good(B))
    mut(B, g)
    lib = B.library()
    rc = lib.bellman_kv_write(g["pkn"], g["pvn"], g["k"], g["v"], g["bt"], g["sl"], g["qs"], None)
    assert rc == code
    assert msg in B.last_error()


PROBE_CASES = [
    ("null pool", dict(pool=None), ERR_INVALID, "device pointers"),
    ("null sink", dict(sink=None), ERR_INVALID, "device pointers"),
    ("tile size", dict(tile=1024), ERR_UNSUPPORTED, "tile_bytes"),
    ("not a multiple", dict(nbytes=4096 * 3 + 8), ERR_INVALID, "multiple"),
    ("not a power of two", dict(nbytes=4096 * 3), ERR_INVALID, "power of two"),
    ("misaligned pool", dict(pool=FAKE + 8), ERR_UNSUPPORTED, "aligned"),
    ("negative waves", dict(waves=-1), ERR_INVALID, "max_waves"),
]


@pytest.mark.parametrize("name,kw,code,msg", PROBE_CASES, ids=[c[0] for c in PROBE_CASES])
def test_probe_rejects(B, name, kw, code, msg):
    a = dict(pool=FAKE, nbytes=4096 * 4, tile=4096, waves=0, sink=FAKE)
    a.update(kw)
    rc = B.library().bellman_probe_gather(a["pool"], a["nbytes"], a["tile"], a["waves"], a["sink"], None)
    assert rc == code
    assert msg in B.last_error()


def test_option_ranges(B):
    g = good(B)
    lib = B.library()
    opts = B.AttnOpts(-1, 0, 0, 0)
    rc = lib.bellman_decode_attention_opts(g["q"], g["k"], g["v"], g["bt"], g["sl"], 0.125, g["out"],
                                           ctypes.byref(opts), None)
    assert rc == ERR_INVALID and "max_waves" in B.last_error()
    for bad_skew in (-2, 256):
        opts = B.AttnOpts(0, bad_skew, 0, 0)
        rc = lib.bellman_decode_attention_opts(g["q"], g["k"], g["v"], g["bt"], g["sl"], 0.125, g["out"],
                                               ctypes.byref(opts), None)
        assert rc == ERR_INVALID and "xcd_skew" in B.last_error()
    for bad_pps in (3, 4):   # 4 is built for fp8 pools only; these are bf16
        opts = B.AttnOpts(0, 0, bad_pps, 0)
        rc = lib.bellman_decode_attention_opts(g["q"], g["k"], g["v"], g["bt"], g["sl"], 0.125, g["out"],
                                               ctypes.byref(opts), None)
        assert rc == ERR_UNSUPPORTED and "pages_per_step" in B.last_error()
    opts = B.AttnOpts(0, 0, 0, 3)
    rc = lib.bellman_decode_attention_opts(g["q"], g["k"], g["v"], g["bt"], g["sl"], 0.125, g["out"],
                                           ctypes.byref(opts), None)
    assert rc == ERR_UNSUPPORTED and "pipeline_depth" in B.last_error()


def test_controller_rejects(B):
    lib = B.library()
    assert not lib.bellman_controller_create(0.1, 0.2, 0, 0.05, 0.2)
    assert not lib.bellman_controller_create(0.1, 0.2, 5, 0.3, 0.2)
    assert not lib.bellman_controller_create(float("nan"), 0.2, 5, 0.05, 0.2)
    assert lib.bellman_length_cap(None) == ERR_INVALID
    c = B.Controller(0.1, 0.2)
    with pytest.raises(B.BellmanError):
        c.length_cap(-1)
    with pytest.raises(B.BellmanError):
        c.length_cap(10, float("inf"))
    with pytest.raises(B.BellmanError):
        B.calibrate_thresholds([])
