"""The prompt path on the GPU against the oracle: the prompt write byte for
byte (pools, lengths, untouched poison), and causal prompt attention element
by element within the bf16 tolerance, on batches that span several 128-row
tiles with ragged tails, chunks after a cached prefix, every GQA group size
the models use, strided rows, empty and malformed requests; at the
6-12k-token prompt sizes on sampled rows."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import paper_2510_15330_amd as bl
from paper_2510_15330_amd import workloads as wl
from tests._gpu import assert_close, bits16

pytestmark = pytest.mark.gpu


def _write(w):
    bl.kv_write(w.k_new, w.v_new, w.k_pages, w.v_pages, w.block_table, w.seq_lens, w.q_start)


def _codes(t):
    # a tensor's elements as host codes: bf16 bits, or fp8 bytes
    return t.cpu().numpy() if t.dtype == torch.uint8 else bits16(t)


def _host_pools(w):
    return _codes(w.k_pages), _codes(w.v_pages)


def _oracle_prefill(w, kp, vp, seq_lens=None, q_bits=None, q_start=None, block_table=None, rows=None):
    fp8 = w.kv == "fp8"
    ks = vs = None
    if fp8:
        # one-token stand-in requests (rows) carry their own request's scales
        pick = slice(None) if rows is None else rows
        ks = w.k_scale.cpu().numpy()[pick]
        vs = w.v_scale.cpu().numpy()[pick]
    return oracle.prefill_attention(
        bits16(w.q) if q_bits is None else q_bits, kp, vp,
        (w.block_table.cpu().numpy() if block_table is None else block_table),
        (w.seq_lens.cpu().numpy().astype(np.int32) if seq_lens is None else seq_lens),
        (w.q_start.cpu().numpy() if q_start is None else q_start), w.scale,
        kv_dtype=oracle.FP8_E4M3FN if fp8 else oracle.BF16, k_scale=ks, v_scale=vs)


def _attend(w, q, out, q_start=None, block_table=None):
    bl.prefill_attention(q, w.k_pages, w.v_pages, w.block_table if block_table is None else block_table,
                         w.seq_lens, w.q_start if q_start is None else q_start, w.scale, out,
                         k_scale=w.k_scale, v_scale=w.v_scale)


def _out_f64(out):
    return out.float().cpu().double().numpy()


# ------------------------------------------------------------- prompt write --

WRITE_CASES = [
    # cached, new, H_kv, D
    ([0, 0, 16, 5], [1, 17, 200, 300], 2, 64),
    ([3, 0, 31], [0, 129, 1], 8, 128),           # an empty request among others
    ([100], [2048], 4, 128),
]


@pytest.mark.parametrize("case", range(len(WRITE_CASES)))
def test_kv_write_bit_exact(case):
    cached, new, H_kv, D = WRITE_CASES[case]
    w = wl.build_prefill(cached=cached, new=new, H_q=H_kv, H_kv=H_kv, D=D, seed=10 + case, device="cuda")
    kp, vp = _host_pools(w)
    seq = w.seq_lens.cpu().numpy().astype(np.int32)
    oracle.kv_write(bits16(w.k_new), bits16(w.v_new), kp, vp, w.block_table.cpu().numpy(), seq,
                    w.q_start.cpu().numpy())
    _write(w)
    assert bl.device_errors() == 0
    gk, gv = _host_pools(w)
    assert np.array_equal(gk, kp) and np.array_equal(gv, vp)
    assert w.seq_lens.cpu().numpy().tolist() == seq.tolist() == (np.array(cached) + np.array(new)).tolist()


def test_kv_write_in_two_chunks_equals_one():
    cached, new = [7, 0], [300, 90]
    w1 = wl.build_prefill(cached=cached, new=new, H_q=8, H_kv=8, D=128, seed=3, device="cuda")
    w2 = wl.build_prefill(cached=cached, new=new, H_q=8, H_kv=8, D=128, seed=3, device="cuda")
    _write(w1)
    # the same tokens as two chunks: 100 + 200 and 50 + 40
    for lo, hi in (((0, 100), (0, 50)), ((100, 300), (50, 90))):
        (a0, a1), (b0, b1) = lo, hi
        rows = torch.cat([torch.arange(a0, a1), 300 + torch.arange(b0, b1)]).cuda()
        qs = torch.tensor([0, a1 - a0, a1 - a0 + b1 - b0], dtype=torch.int32, device="cuda")
        bl.kv_write(w2.k_new[rows], w2.v_new[rows], w2.k_pages, w2.v_pages, w2.block_table, w2.seq_lens, qs)
    assert bl.device_errors() == 0
    assert torch.equal(w1.k_pages.view(torch.int16), w2.k_pages.view(torch.int16))
    assert torch.equal(w1.v_pages.view(torch.int16), w2.v_pages.view(torch.int16))
    assert torch.equal(w1.seq_lens, w2.seq_lens)


def test_kv_write_flags_slots_outside_the_table():
    w = wl.build_prefill(cached=[0, 4], new=[20, 40], H_q=2, H_kv=2, D=64, seed=5, device="cuda", extra_table=0)
    kp0, vp0 = _host_pools(w)
    w.block_table[1, 2] = -1                         # positions 32..43 of request 1 have no page
    _write(w)
    assert bl.device_errors() == 1
    assert w.seq_lens.cpu().tolist() == [20, 44]     # every position lies inside the table's width
    w2 = wl.build_prefill(cached=[0, 4], new=[20, 40], H_q=2, H_kv=2, D=64, seed=5, device="cuda", extra_table=0)
    w2.seq_lens[1] = 10                              # 10 + 40 = 50 > 3 pages x 16: length left unchanged
    _write(w2)
    assert bl.device_errors() == 1
    assert w2.seq_lens.cpu().tolist() == [20, 10]
    gk, _ = _host_pools(w2)
    assert not np.array_equal(gk, kp0)               # the positions that fit were still written


# --------------------------------------------------------- prompt attention --

ATTN_CASES = [
    # name, cached, new, H_q, H_kv, D
    ("tiny_d64_g4", [0, 0, 16, 5], [1, 17, 200, 300], 8, 2, 64),
    ("ragged_d128_g4", [0, 0, 0, 0, 0], [128, 129, 257, 31, 500], 32, 8, 128),
    ("chunk_after_prefix", [33, 700, 1, 16], [9, 300, 64, 128], 16, 4, 128),
    ("g1_d128", [5, 0], [140, 260], 4, 4, 128),
    ("g8_d128", [0, 200], [333, 77], 64, 8, 128),
    ("g16_d64", [40, 0], [200, 129], 32, 2, 64),
    ("empty_requests", [10, 0, 3, 0], [0, 150, 0, 1], 8, 2, 128),
]


# fp8 pools: the codes widen to bf16 exactly and the scales enter in fp32,
# so the arithmetic is the bf16 path's and so is the tolerance
@pytest.mark.parametrize("kv", ["bf16", "fp8"])
@pytest.mark.parametrize("case", ATTN_CASES, ids=[c[0] for c in ATTN_CASES])
def test_prefill_matches_oracle(case, kv):
    name, cached, new, H_q, H_kv, D = case
    w = wl.build_prefill(cached=cached, new=new, H_q=H_q, H_kv=H_kv, D=D, seed=len(name), device="cuda", kv=kv)
    _write(w)
    out = torch.full((w.T, H_q, D), float("nan"), dtype=torch.bfloat16, device="cuda")
    _attend(w, w.q, out)
    assert bl.device_errors() == 0
    kp, vp = _host_pools(w)
    ref = _oracle_prefill(w, kp, vp)
    assert_close(_out_f64(out), ref, "bf16", f"{name} {kv}")


@pytest.mark.parametrize("kv", ["bf16", "fp8"])
def test_prefill_negative_zero_and_sharp_scales(kv):
    # any finite softmax scale: negative (the kernel flips the query's signs),
    # zero (uniform weights over each row's visible keys) and four times the
    # usual 1/sqrt(D) (much sharper weights leave single value rows, whose
    # own bf16 rounding reaches the max-abs bound)
    cached, new, H_q, H_kv, D = [0, 40], [150, 90], 8, 2, 128
    for scale in (-0.0884, 0.0, 0.3536):
        w = wl.build_prefill(cached=cached, new=new, H_q=H_q, H_kv=H_kv, D=D, seed=77, device="cuda", kv=kv)
        w.scale = scale
        _write(w)
        out = torch.full((w.T, H_q, D), float("nan"), dtype=torch.bfloat16, device="cuda")
        _attend(w, w.q, out)
        assert bl.device_errors() == 0
        kp, vp = _host_pools(w)
        assert_close(_out_f64(out), _oracle_prefill(w, kp, vp), "bf16", f"scale {scale} {kv}")


def test_prefill_value_magnitudes():
    # bf16 values of each KV head at their own magnitude, 2^-100 to 2^16
    # (past fp16's range): the fp16 value copy's per-head power-of-two scale
    # keeps each head's output, divided by its factor, within the bound
    factors = [2.0 ** 16, 2.0 ** -24, 1.0, 2.0 ** -100]
    cached, new, H_q, H_kv, D = [20, 0, 300], [100, 70, 45], 8, 4, 128
    w = wl.build_prefill(cached=cached, new=new, H_q=H_q, H_kv=H_kv, D=D, seed=5, device="cuda")
    fac = torch.tensor(factors, dtype=torch.float32, device="cuda")
    # powers of two: exact in bf16, and NaN poison stays NaN
    w.v_pages.copy_((w.v_pages.float() * fac.view(1, H_kv, 1, 1)).to(torch.bfloat16))
    w.v_new.copy_((w.v_new.float() * fac.view(1, H_kv, 1)).to(torch.bfloat16))
    _write(w)
    out = torch.full((w.T, H_q, D), float("nan"), dtype=torch.bfloat16, device="cuda")
    _attend(w, w.q, out)
    assert bl.device_errors() == 0
    kp, vp = _host_pools(w)
    ref = _oracle_prefill(w, kp, vp)
    got = _out_f64(out)
    G = H_q // H_kv
    per_head = np.repeat(np.array(factors), G)[None, :, None]
    assert_close(got / per_head, ref / per_head, "bf16", "per-head magnitudes")


def _sweep_counts(rng, B, edge):
    out = []
    for _ in range(B):
        kind = rng.integers(0, 4)
        if kind == 0:
            out.append(0)
        elif kind == 1:
            out.append(int(edge * rng.integers(1, 6) + rng.integers(-1, 2)))
        else:
            out.append(int(rng.integers(1, 400)))
    return out


@pytest.mark.parametrize("seed", range(12))
def test_prefill_random_sweep(seed):
    # seeded shapes: GQA group, head_dim, cached prefixes and new-token counts
    # on and next to page (16), step (64) and tile (128) edges, empty chunks
    rng = np.random.default_rng(7000 + seed)
    kv = "fp8" if seed % 3 == 2 else "bf16"
    H_kv = int(rng.choice([1, 2, 4, 8]))
    G = int(rng.choice([1, 2, 3, 4, 8, 16]))
    D = 64 if seed % 2 else 128
    B = int(rng.integers(1, 7))
    cached = _sweep_counts(rng, B, 16)
    new = _sweep_counts(rng, B, int(rng.choice([16, 64, 128])))
    w = wl.build_prefill(cached=cached, new=new, H_q=G * H_kv, H_kv=H_kv, D=D, seed=7000 + seed, device="cuda",
                         kv=kv)
    kp0, vp0 = _host_pools(w)
    sl0 = w.seq_lens.cpu().numpy().astype(np.int32)
    _write(w)
    assert bl.device_errors() == 0
    kp, vp = _host_pools(w)
    kx, vx, sx = kp0.copy(), vp0.copy(), sl0.copy()
    oracle.kv_write(_codes(w.k_new), _codes(w.v_new), kx, vx, w.block_table.cpu().numpy(), sx,
                    w.q_start.cpu().numpy(), kv_dtype=oracle.FP8_E4M3FN if kv == "fp8" else oracle.BF16)
    what = f"seed={seed} {kv} G={G} H_kv={H_kv} D={D} cached={cached} new={new}"
    assert np.array_equal(kp, kx) and np.array_equal(vp, vx), what
    if w.T == 0:
        return
    out = torch.full((w.T, G * H_kv, D), float("nan"), dtype=torch.bfloat16, device="cuda")
    _attend(w, w.q, out)
    assert bl.device_errors() == 0
    assert_close(_out_f64(out), _oracle_prefill(w, kp, vp), "bf16", what)


def test_prefill_many_requests():
    # 1500 short requests (many with nothing cached or nothing new): the
    # write's and the attention's planners scan the batch in several chunks
    rng = np.random.default_rng(1500)
    B = 1500
    cached = [int(x) for x in rng.integers(0, 40, size=B) * (rng.random(B) < 0.7)]
    new = [int(x) for x in rng.integers(0, 21, size=B) * (rng.random(B) < 0.8)]
    w = wl.build_prefill(cached=cached, new=new, H_q=8, H_kv=2, D=64, seed=1500, device="cuda")
    kp0, vp0 = _host_pools(w)
    sl0 = w.seq_lens.cpu().numpy().astype(np.int32)
    _write(w)
    assert bl.device_errors() == 0
    kp, vp = _host_pools(w)
    kx, vx, sx = kp0.copy(), vp0.copy(), sl0.copy()
    oracle.kv_write(bits16(w.k_new), bits16(w.v_new), kx, vx, w.block_table.cpu().numpy(), sx, w.q_start.cpu().numpy())
    assert np.array_equal(kp, kx) and np.array_equal(vp, vx), "prompt write bytes"
    assert np.array_equal(w.seq_lens.cpu().numpy(), sx)
    out = torch.full((w.T, 8, 64), float("nan"), dtype=torch.bfloat16, device="cuda")
    bl.prefill_attention(w.q, w.k_pages, w.v_pages, w.block_table, w.seq_lens, w.q_start, w.scale, out)
    assert bl.device_errors() == 0
    assert_close(_out_f64(out), _oracle_prefill(w, kp, vp), "bf16", "1500 requests")


def test_prefill_strided_rows():
    # q and out as column slices of wider tensors (row strides above H * D)
    cached, new, H_q, H_kv, D = [3, 0], [150, 40], 8, 2, 128
    w = wl.build_prefill(cached=cached, new=new, H_q=H_q, H_kv=H_kv, D=D, seed=21, device="cuda")
    _write(w)
    T = w.T
    qwide = torch.zeros((T, H_q + 3, D), dtype=torch.bfloat16, device="cuda")
    qwide[:, 1:1 + H_q] = w.q
    owide = torch.full((T, H_q + 5, D), 7.0, dtype=torch.bfloat16, device="cuda")
    bl.prefill_attention(qwide[:, 1:1 + H_q], w.k_pages, w.v_pages, w.block_table, w.seq_lens, w.q_start,
                         w.scale, owide[:, 2:2 + H_q])
    assert bl.device_errors() == 0
    kp, vp = _host_pools(w)
    assert_close(_out_f64(owide[:, 2:2 + H_q]), _oracle_prefill(w, kp, vp), "bf16", "strided")
    assert (owide[:, :2] == 7).all() and (owide[:, 2 + H_q:] == 7).all()


def test_prefill_flags_malformed_requests():
    cached, new, H_q, H_kv, D = [0, 0, 0], [100, 50, 70], 8, 2, 64
    w = wl.build_prefill(cached=cached, new=new, H_q=H_q, H_kv=H_kv, D=D, seed=31, device="cuda")
    _write(w)
    kp, vp = _host_pools(w)
    ref = _oracle_prefill(w, kp, vp)
    # request 1 claims more query tokens than it holds: flagged, its rows untouched
    w.seq_lens[1] = 20
    out = torch.full((w.T, H_q, D), 3.0, dtype=torch.bfloat16, device="cuda")
    bl.prefill_attention(w.q, w.k_pages, w.v_pages, w.block_table, w.seq_lens, w.q_start, w.scale, out)
    assert bl.device_errors() == 2
    o = _out_f64(out)
    assert (o[100:150] == 3.0).all()
    assert_close(np.concatenate([o[:100], o[150:]]), np.concatenate([ref[:100], ref[150:]]), "bf16", "others")
    # a decreasing q_start: nothing is written
    w.seq_lens[1] = 50
    bad = torch.tensor([0, 100, 90, 220], dtype=torch.int32, device="cuda")
    out.fill_(3.0)
    bl.prefill_attention(w.q, w.k_pages, w.v_pages, w.block_table, w.seq_lens, bad, w.scale, out)
    assert bl.device_errors() == 2
    assert (out == 3.0).all()
    # a table entry outside the pool: flagged (page skipped), no fault
    bt = w.block_table.clone()
    bt[2, 1] = w.num_pages + 1000
    bl.prefill_attention(w.q, w.k_pages, w.v_pages, bt, w.seq_lens, w.q_start, w.scale, out)
    assert bl.device_errors() == 4
    assert_close(_out_f64(out)[:150], ref[:150], "bf16", "requests with good tables")


def test_prefill_empty_batch_and_rejections():
    w = wl.build_prefill(cached=[4], new=[0], H_q=4, H_kv=2, D=64, seed=1, device="cuda")
    out = torch.empty((0, 4, 64), dtype=torch.bfloat16, device="cuda")
    bl.prefill_attention(w.q, w.k_pages, w.v_pages, w.block_table, w.seq_lens, w.q_start, w.scale, out)
    assert bl.device_errors() == 0
    # fp8 pools: an empty batch is accepted; pools without their scales are not
    kp8 = torch.zeros((4, 2, 4, 16, 16), dtype=torch.uint8, device="cuda")
    vp8 = torch.zeros((4, 2, 64, 16), dtype=torch.uint8, device="cuda")
    s = torch.ones((1, 2), dtype=torch.float32, device="cuda")
    lib = bl.library()
    from paper_2510_15330_amd import _binding as B
    rc = lib.bellman_prefill_attention(B.desc(w.q), B.desc(kp8, s), B.desc(vp8, s), B.desc(w.block_table),
                                       B.desc(w.seq_lens), B.desc(w.q_start), 0.125, B.desc(out), None)
    assert rc == 0
    rc = lib.bellman_prefill_attention(B.desc(w.q), B.desc(kp8), B.desc(vp8), B.desc(w.block_table),
                                       B.desc(w.seq_lens), B.desc(w.q_start), 0.125, B.desc(out), None)
    assert rc == -1 and "dequant_scale" in bl.last_error()
    torch.cuda.synchronize()
    assert bl.device_errors() == 0


# ------------------------------------------------------------ full sizes --

def _sampled_rows(w, rng, per_request):
    """(token index, request, position) of sampled query rows: each request's
    first and last rows, rows on both sides of 128-row tile edges, and random
    ones."""
    picks = []
    qs = w.q_start.cpu().numpy()
    for b in range(w.B):
        n = int(w.new[b])
        if n == 0:
            continue
        rows = {0, n - 1, min(127, n - 1), min(128, n - 1)}
        rows |= set(rng.integers(0, n, size=per_request).tolist())
        for i in sorted(rows):
            picks.append((int(qs[b]) + i, b, int(w.cached[b]) + i))
    return picks


@pytest.mark.parametrize("name,kv", [("prefill_summarization", "bf16"), ("prefill_chunked", "bf16"),
                                     ("prefill_summarization", "fp8")])
def test_prefill_full_size_sampled_rows(name, kv):
    w = wl.build_prefill(name, seed=0, device="cuda", kv=kv)
    _write(w)
    out = torch.empty((w.T, w.H_q, w.D), dtype=torch.bfloat16, device="cuda")
    _attend(w, w.q, out)
    assert bl.device_errors() == 0
    assert torch.isfinite(out).all()
    picks = _sampled_rows(w, np.random.default_rng(7), 3)
    # the oracle takes each sampled row as a one-token request whose length
    # ends at the row's position, over the same pages
    rows = [p[0] for p in picks]
    bt = w.block_table.cpu().numpy()[[p[1] for p in picks]]
    lens = np.array([p[2] + 1 for p in picks], dtype=np.int32)
    q_bits = bits16(w.q[torch.tensor(rows, device="cuda")])
    kp, vp = _host_pools(w)
    ref = _oracle_prefill(w, kp, vp, seq_lens=lens, q_bits=q_bits,
                          q_start=np.arange(len(rows) + 1, dtype=np.int32), block_table=bt,
                          rows=[p[1] for p in picks])
    assert_close(_out_f64(out)[rows], ref, "bf16", f"{name} {kv}")


def test_kv_write_fp8_codes_bit_exact():
    # 1-byte pools (fp8 codes, copied as bytes): random codes everywhere,
    # four requests with unaligned cached prefixes
    rng = np.random.default_rng(44)
    B, H_kv, D = 4, 2, 128
    cached, new = np.array([3, 0, 17, 40]), np.array([29, 16, 1, 70])
    need = (cached + new + 15) // 16
    NP = int(need.sum()) + 4
    perm = rng.permutation(NP).astype(np.int32)
    bt = np.full((B, int(need.max()) + 1), -1, dtype=np.int32)
    pos = 0
    for b in range(B):
        bt[b, :need[b]] = perm[pos:pos + need[b]]
        pos += need[b]
    kp = rng.integers(0, 256, size=(NP, H_kv, D // 16, 16, 16), dtype=np.uint8)
    vp = rng.integers(0, 256, size=(NP, H_kv, D, 16), dtype=np.uint8)
    T = int(new.sum())
    kn = rng.integers(0, 256, size=(T, H_kv, D), dtype=np.uint8)
    vn = rng.integers(0, 256, size=(T, H_kv, D), dtype=np.uint8)
    qs = np.concatenate([[0], np.cumsum(new)]).astype(np.int32)
    sl = cached.astype(np.int32)
    # every device tensor stays referenced until the call has run (a
    # descriptor holds only the pointer)
    gk, gv, gsl = (torch.from_numpy(x).cuda() for x in (kp, vp, sl))
    gkn, gvn, gbt, gqs = (torch.from_numpy(x).cuda() for x in (kn, vn, bt, qs))
    bl.kv_write(gkn, gvn, gk, gv, gbt, gsl, gqs)
    torch.cuda.synchronize()
    assert bl.device_errors() == 0
    ek, ev, esl = kp.copy(), vp.copy(), sl.copy()
    oracle.kv_write(kn, vn, ek, ev, bt, esl, qs, kv_dtype=oracle.FP8_E4M3FN)
    assert np.array_equal(gk.cpu().numpy(), ek) and np.array_equal(gv.cpu().numpy(), ev)
    assert gsl.cpu().tolist() == esl.tolist() == (cached + new).tolist()
