"""Seeded synthetic decode-step inputs.

This module draws inputs only: request lengths, page placement, bf16/fp8
values and poison.  It holds none of the attention arithmetic, so both the
GPU tests and the CPU oracle may take their inputs from it.

The paper's setting (beLLMan, Sec. 3 "Setup and trace") summarises 6- and
12-page papers with a 27B model under a Poisson request trace, and caps the
output length of each request under congestion (Sec. 3 "Our key proposal").
Neither the papers, the model nor the traces are available; the workloads
below stand in for them with the shapes and length laws of the decode batches
that setting produces:

* ``tiny``                 B=3, KV lengths {1, 17, 200} after one append,
                           8 query / 2 KV heads, head_dim 64, 64-page pool.
* ``llama3_8b``            B=64, 32/8 heads, head_dim 128, lengths U{1024..4096},
                           100 decode steps.
* ``summarization``        B=256, 32/8 heads, head_dim 128; length = prompt
                           U{6000..12000} + generated floor(LogNormal(ln 500,
                           0.5)) clipped to [1, 1500]; 50 decode steps.
* ``summarization_capped`` as above, generated length capped per request at a
                           target drawn from {100, 200, 400}.
* ``stress_fp8``           B=512, 64/8 heads, head_dim 128, lengths drawn from
                           P(L = k) proportional to k^-1.2 on [128, 32768],
                           fp8-e4m3fn K/V with one fp32 scale per (request, KV
                           head) for K and one for V.

Prompt (prefill) batches, drawn by ``build_prefill``:

* ``prefill_tiny``          4 requests, 8 query / 2 KV heads, head_dim 64,
                           cached {0, 0, 16, 5} + new {1, 17, 200, 300} tokens.
* ``prefill_summarization`` 4 whole prompts of U{6000..12000} tokens,
                           32/8 heads, head_dim 128.
* ``prefill_chunked``       the last 2048 tokens of 4 such prompts (the rest
                           cached), the chunk size of the serving model.

Values are N(0, 1) rounded to bf16.  Pages (16 tokens) are scattered over a
randomly permuted pool, every page a request will need during the run is
reserved up front, slots that hold no token yet and pages that belong to no
request hold NaN, and unused block-table entries hold -1.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np
import torch

PAGE = 16
BF16_NAN_BITS = 0x7FC0
FP8_NAN_CODE = 0x7F
FP8_MAX = 448.0

CONFIGS = {
    "tiny": dict(B=3, H_q=8, H_kv=2, D=64, kv="bf16", steps=1),
    "llama3_8b": dict(B=64, H_q=32, H_kv=8, D=128, kv="bf16", steps=100),
    "summarization": dict(B=256, H_q=32, H_kv=8, D=128, kv="bf16", steps=50),
    "summarization_capped": dict(B=256, H_q=32, H_kv=8, D=128, kv="bf16", steps=50),
    "stress_fp8": dict(B=512, H_q=64, H_kv=8, D=128, kv="fp8", steps=50),
}

PREFILL_CONFIGS = {
    "prefill_tiny": dict(H_q=8, H_kv=2, D=64),
    "prefill_summarization": dict(H_q=32, H_kv=8, D=128),
    "prefill_chunked": dict(H_q=32, H_kv=8, D=128),
}

# Seed-stream indices under numpy's SeedSequence(seed).spawn(...)
_S_LEN, _S_GEN, _S_CAP, _S_PAGES, _S_VALUES, _S_P_LEN, _S_P_PAGES, _S_P_VALUES = range(8)


def _streams(seed):
    return np.random.SeedSequence(seed).spawn(8)


def sample_lengths(name, seed=0, tiny_reading="after"):
    """KV lengths before the first append of the run, int64 [B].

    For ``tiny`` the lengths {1, 17, 200} are read as the lengths *after* the
    step's append (pre-append {0, 16, 199}); ``tiny_reading="before"`` gives
    the other reading (pre-append {1, 17, 200}).  For ``stress_fp8`` the drawn
    lengths are attention lengths of the first step (pre-append L - 1).
    Returns (lens0, info) where info carries the generated lengths and caps of
    the summarization workloads.
    """
    ss = _streams(seed)
    info = {}
    if name == "tiny":
        lens = np.array([1, 17, 200], dtype=np.int64)
        return (lens - 1 if tiny_reading == "after" else lens), info
    if name == "llama3_8b":
        rng = np.random.default_rng(ss[_S_LEN])
        return rng.integers(1024, 4096, size=64, endpoint=True).astype(np.int64), info
    if name in ("summarization", "summarization_capped"):
        B = 256
        prompt = np.random.default_rng(ss[_S_LEN]).integers(6000, 12000, size=B, endpoint=True)
        z = np.random.default_rng(ss[_S_GEN]).standard_normal(B)
        gen = np.clip(np.floor(np.exp(math.log(500.0) + 0.5 * z)), 1, 1500).astype(np.int64)
        info["prompt"] = prompt.astype(np.int64)
        info["generated"] = gen
        if name == "summarization_capped":
            cap = np.random.default_rng(ss[_S_CAP]).choice(np.array([100, 200, 400]), size=B)
            info["cap"] = cap.astype(np.int64)
            gen = np.minimum(gen, cap)
            info["generated_capped"] = gen
        return (prompt + gen).astype(np.int64), info
    if name == "stress_fp8":
        ks = np.arange(128, 32768 + 1, dtype=np.int64)
        w = ks.astype(np.float64) ** -1.2
        L = np.random.default_rng(ss[_S_LEN]).choice(ks, size=512, p=w / w.sum())
        return (L - 1).astype(np.int64), info
    raise KeyError(name)


@dataclasses.dataclass
class Workload:
    name: str
    B: int
    H_q: int
    H_kv: int
    D: int
    kv: str                      # "bf16" or "fp8"
    steps: int
    scale: float                 # fp32 softmax scale 1/sqrt(D)
    lens0: np.ndarray            # int64 [B], KV lengths before the first append
    num_pages: int
    block_table: torch.Tensor    # int32 [B, maxP]
    seq_lens: torch.Tensor       # int32 [B], initialised to lens0
    k_pages: torch.Tensor        # [NP, H_kv, D/x, 16, x]  bf16 or uint8 codes
    v_pages: torch.Tensor        # [NP, H_kv, D, 16]
    q: torch.Tensor              # bf16 [steps, B, H_q, D]
    k_new: torch.Tensor          # [steps, B, H_kv, D] bf16 or uint8 codes
    v_new: torch.Tensor
    k_scale: torch.Tensor | None  # fp32 [B, H_kv] (fp8 only)
    v_scale: torch.Tensor | None
    info: dict

    @property
    def x(self):
        return 8 if self.kv == "bf16" else 16

    @property
    def max_pages(self):
        return int(self.block_table.shape[1])

    def elem_bytes(self):
        return 2 if self.kv == "bf16" else 1

    def lens_at(self, step):
        """Attention lengths of decode step ``step`` (after its append)."""
        return self.lens0 + step + 1

    def kv_bytes(self, step):
        """K+V bytes the attention of ``step`` must read (tokens in use)."""
        return int(self.lens_at(step).sum()) * self.H_kv * self.D * 2 * self.elem_bytes()

    def algorithmic_bytes(self, step):
        """All bytes one decode-attention launch must touch at least once."""
        L = self.lens_at(step)
        pages = int(((L + PAGE - 1) // PAGE).sum())
        qo = 2 * self.B * self.H_q * self.D * 2
        scales = 2 * self.B * self.H_kv * 4 if self.kv == "fp8" else 0
        return self.kv_bytes(step) + qo + pages * 4 + self.B * 4 + scales

    def append_bytes(self):
        """Bytes one KV append reads and writes (new rows in, pool slots out)."""
        return 2 * 2 * self.B * self.H_kv * self.D * self.elem_bytes() + 2 * self.B * 4

    def flops(self, step):
        """Multiply-adds of QK^T and PV, two flops each."""
        return 4 * self.D * self.H_q * int(self.lens_at(step).sum())


def _bf16_normal(shape, gen, device):
    """N(0, 1) float32 draws rounded to bf16 (torch's round-to-nearest-even)."""
    return torch.randn(shape, generator=gen, device=device, dtype=torch.float32).to(torch.bfloat16)


def build(name, seed=0, device="cpu", steps=None, tiny_reading="after", slack_pages=None):
    """Materialise a workload on ``device``.

    ``steps`` is the number of decode steps the caller will run from the
    initial state; pages are reserved for all of them.
    """
    cfg = CONFIGS[name]
    B, H_q, H_kv, D, kv = cfg["B"], cfg["H_q"], cfg["H_kv"], cfg["D"], cfg["kv"]
    steps = cfg["steps"] if steps is None else int(steps)
    lens0, info = sample_lengths(name, seed, tiny_reading)
    ss = _streams(seed)

    final = lens0 + steps
    need = (final + PAGE - 1) // PAGE
    total = int(need.sum())
    if name == "tiny":
        NP = 64
    else:
        NP = total + (slack_pages if slack_pages is not None else max(64, total // 64))
    assert NP >= total
    perm = np.random.default_rng(ss[_S_PAGES]).permutation(NP).astype(np.int32)
    maxP = int(need.max())
    bt = np.full((B, maxP), -1, dtype=np.int32)
    owner = np.full(NP, -1, dtype=np.int64)
    logical = np.zeros(NP, dtype=np.int64)
    pos = 0
    for b in range(B):
        n = int(need[b])
        pages = perm[pos:pos + n]
        bt[b, :n] = pages
        owner[pages] = b
        logical[pages] = np.arange(n)
        pos += n
    # tokens already present in each page at the start of the run
    filled = np.where(owner >= 0, np.clip(lens0[np.maximum(owner, 0)] - PAGE * logical, 0, PAGE), 0)

    gen = torch.Generator(device=device)
    gen.manual_seed(int(ss[_S_VALUES].generate_state(1, dtype=np.uint64)[0] & 0x7FFFFFFFFFFFFFFF))

    x = 8 if kv == "bf16" else 16
    kshape = (NP, H_kv, D // x, PAGE, x)
    vshape = (NP, H_kv, D, PAGE)
    filled_t = torch.from_numpy(filled).to(device)
    slot = torch.arange(PAGE, device=device)
    live = slot[None, :] < filled_t[:, None]                    # [NP, 16]
    kmask = live[:, None, None, :, None]
    vmask = live[:, None, None, :]

    q = _bf16_normal((steps, B, H_q, D), gen, device)
    scale = float(np.float32(1.0 / math.sqrt(D)))

    if kv == "bf16":
        k_pages = _fill_pages(kshape, gen, device)
        v_pages = _fill_pages(vshape, gen, device)
        nan = torch.tensor(BF16_NAN_BITS, dtype=torch.int16, device=device).view(torch.bfloat16)
        k_pages = torch.where(kmask, k_pages, nan)
        v_pages = torch.where(vmask, v_pages, nan)
        k_new = _bf16_normal((steps, B, H_kv, D), gen, device)
        v_new = _bf16_normal((steps, B, H_kv, D), gen, device)
        k_scale = v_scale = None
    else:
        owner_t = torch.from_numpy(owner).to(device)
        k_pages, k_scale = _fp8_pool(kshape, gen, device, kmask, owner_t, B, H_kv, (2, 3, 4))
        v_pages, v_scale = _fp8_pool(vshape, gen, device, vmask, owner_t, B, H_kv, (2, 3))
        k_new = _fp8_quantise(torch.randn((steps, B, H_kv, D), generator=gen, device=device),
                              k_scale[None, :, :, None])
        v_new = _fp8_quantise(torch.randn((steps, B, H_kv, D), generator=gen, device=device),
                              v_scale[None, :, :, None])

    return Workload(
        name=name, B=B, H_q=H_q, H_kv=H_kv, D=D, kv=kv, steps=steps, scale=scale,
        lens0=lens0, num_pages=NP,
        block_table=torch.from_numpy(bt).to(device),
        seq_lens=torch.from_numpy(lens0.astype(np.int32)).to(device),
        k_pages=k_pages.contiguous(), v_pages=v_pages.contiguous(), q=q,
        k_new=k_new, v_new=v_new, k_scale=k_scale, v_scale=v_scale, info=info)


def _fill_pages(shape, gen, device, chunk_pages=4096):
    out = torch.empty(shape, dtype=torch.bfloat16, device=device)
    for p0 in range(0, shape[0], chunk_pages):
        p1 = min(shape[0], p0 + chunk_pages)
        out[p0:p1] = _bf16_normal((p1 - p0,) + tuple(shape[1:]), gen, device)
    return out


def _fp8_quantise(x, s):
    """Round x / s to e4m3fn with saturation at +-448 (the cast alone does not saturate)."""
    y = (x / s).clamp(-FP8_MAX, FP8_MAX).to(torch.float8_e4m3fn)
    return y.view(torch.uint8)


def _fp8_pool(shape, gen, device, mask, owner, B, H_kv, red_dims, chunk_pages=4096):
    """Draw N(0,1) values per page, choose scale = amax / 448 per (request, head)
    over the tokens present, and store e4m3fn codes (NaN in empty slots)."""
    NP = shape[0]
    vals = torch.empty(shape, dtype=torch.float32, device=device)
    for p0 in range(0, NP, chunk_pages):
        p1 = min(NP, p0 + chunk_pages)
        vals[p0:p1] = torch.randn((p1 - p0,) + tuple(shape[1:]), generator=gen, device=device)
    page_amax = torch.where(mask, vals.abs(), torch.zeros((), device=device)).amax(dim=red_dims)
    amax = torch.zeros((B, H_kv), dtype=torch.float32, device=device)
    own = owner >= 0
    idx = owner.clamp(min=0)[:, None].expand(NP, H_kv)
    amax.scatter_reduce_(0, idx[own], page_amax[own], reduce="amax")
    scale = torch.where(amax > 0, amax / FP8_MAX, torch.ones_like(amax))
    page_scale = torch.where(own[:, None], scale[owner.clamp(min=0)], torch.ones((), device=device))
    bshape = (NP, H_kv) + (1,) * (len(shape) - 2)
    codes = torch.empty(shape, dtype=torch.uint8, device=device)
    for p0 in range(0, NP, chunk_pages):
        p1 = min(NP, p0 + chunk_pages)
        codes[p0:p1] = _fp8_quantise(vals[p0:p1], page_scale[p0:p1].view((p1 - p0,) + bshape[1:]))
    del vals
    codes = torch.where(mask, codes, torch.tensor(FP8_NAN_CODE, dtype=torch.uint8, device=device))
    return codes, scale.contiguous()


# ------------------------------------------------------------ prompt batches --

@dataclasses.dataclass
class PrefillWorkload:
    name: str
    H_q: int
    H_kv: int
    D: int
    scale: float                 # fp32 softmax scale 1/sqrt(D)
    cached: np.ndarray           # int64 [B], tokens already in the cache
    new: np.ndarray              # int64 [B], prompt tokens of this batch
    num_pages: int
    block_table: torch.Tensor    # int32 [B, maxP]
    seq_lens: torch.Tensor       # int32 [B], initialised to ``cached``
    q_start: torch.Tensor        # int32 [B + 1], exclusive prefix sum of ``new``
    k_pages: torch.Tensor        # bf16 [NP, H_kv, D/8, 16, 8]
    v_pages: torch.Tensor        # bf16 [NP, H_kv, D, 16]
    q: torch.Tensor              # bf16 [T, H_q, D]
    k_new: torch.Tensor          # bf16 [T, H_kv, D] (fp8 pools: e4m3fn codes, uint8)
    v_new: torch.Tensor
    kv: str = "bf16"             # "bf16", or "fp8": pools [NP, H_kv, D/16, 16, 16] / [NP, H_kv, D, 16] of codes
    k_scale: torch.Tensor = None  # fp8 only: fp32 [B, H_kv] dequantisation scales
    v_scale: torch.Tensor = None

    @property
    def B(self):
        return len(self.new)

    @property
    def T(self):
        return int(self.new.sum())

    def total(self):
        return self.cached + self.new

    def flops(self):
        """Multiply-adds of QK^T and PV over the visible (causal) pairs, two
        flops each: query i of request b sees cached_b + i + 1 keys."""
        c, n = self.cached.astype(np.int64), self.new.astype(np.int64)
        pairs = int((n * c + n * (n + 1) // 2).sum())
        return 4 * self.D * self.H_q * pairs

    def write_bytes(self):
        """Bytes one prompt write moves (new rows in, pool slots out)."""
        return 2 * 2 * self.T * self.H_kv * self.D * 2


def prefill_lengths(name, seed=0):
    """(cached, new) token counts, int64 [B] each."""
    ss = _streams(seed)
    if name == "prefill_tiny":
        return np.array([0, 0, 16, 5], dtype=np.int64), np.array([1, 17, 200, 300], dtype=np.int64)
    prompt = np.random.default_rng(ss[_S_P_LEN]).integers(6000, 12000, size=4, endpoint=True).astype(np.int64)
    if name == "prefill_summarization":
        return np.zeros(4, dtype=np.int64), prompt
    if name == "prefill_chunked":
        return prompt - 2048, np.full(4, 2048, dtype=np.int64)
    raise KeyError(name)


def build_prefill(name=None, seed=0, device="cpu", cached=None, new=None, H_q=None, H_kv=None, D=None,
                  slack_pages=5, extra_table=1, kv="bf16"):
    """Materialise a prompt batch on ``device``: pages for every cached and new
    token (scattered over a permuted pool), cached tokens' K/V present, every
    other slot NaN, unused table entries -1.  Named configurations come from
    PREFILL_CONFIGS / prefill_lengths; explicit ``cached``/``new`` and head
    counts override them."""
    if name is not None:
        cfg = PREFILL_CONFIGS[name]
        c0, n0 = prefill_lengths(name, seed)
        cached = c0 if cached is None else cached
        new = n0 if new is None else new
        H_q, H_kv, D = (cfg["H_q"] if H_q is None else H_q, cfg["H_kv"] if H_kv is None else H_kv,
                        cfg["D"] if D is None else D)
    cached = np.asarray(cached, dtype=np.int64)
    new = np.asarray(new, dtype=np.int64)
    B = len(new)
    ss = _streams(seed)
    final = cached + new
    need = (final + PAGE - 1) // PAGE
    NP = int(need.sum()) + slack_pages
    perm = np.random.default_rng(ss[_S_P_PAGES]).permutation(NP).astype(np.int32)
    maxP = int(need.max()) + extra_table if B else 1
    bt = np.full((B, maxP), -1, dtype=np.int32)
    owner = np.full(NP, -1, dtype=np.int64)
    logical = np.zeros(NP, dtype=np.int64)
    pos = 0
    for b in range(B):
        n = int(need[b])
        pages = perm[pos:pos + n]
        bt[b, :n] = pages
        owner[pages] = b
        logical[pages] = np.arange(n)
        pos += n
    filled = np.where(owner >= 0, np.clip(cached[np.maximum(owner, 0)] - PAGE * logical, 0, PAGE), 0)

    gen = torch.Generator(device=device)
    gen.manual_seed(int(ss[_S_P_VALUES].generate_state(1, dtype=np.uint64)[0] & 0x7FFFFFFFFFFFFFFF))
    filled_t = torch.from_numpy(filled).to(device)
    slot = torch.arange(PAGE, device=device)
    live = slot[None, :] < filled_t[:, None]
    T = int(new.sum())
    q_start = np.concatenate([[0], np.cumsum(new)]).astype(np.int32)
    k_scale = v_scale = None
    if kv == "bf16":
        kshape = (NP, H_kv, D // 8, PAGE, 8)
        vshape = (NP, H_kv, D, PAGE)
        nan = torch.tensor(BF16_NAN_BITS, dtype=torch.int16, device=device).view(torch.bfloat16)
        k_pages = torch.where(live[:, None, None, :, None], _fill_pages(kshape, gen, device), nan)
        v_pages = torch.where(live[:, None, None, :], _fill_pages(vshape, gen, device), nan)
        q = _bf16_normal((T, H_q, D), gen, device)
        k_new = _bf16_normal((T, H_kv, D), gen, device)
        v_new = _bf16_normal((T, H_kv, D), gen, device)
    else:
        # codes of N(0,1) values at scale = amax / 448 of each (request, head)'s
        # cached tokens (1 where none is cached); the new tokens' codes at the
        # same scales, as a quantising writer would store them
        kshape = (NP, H_kv, D // 16, PAGE, 16)
        vshape = (NP, H_kv, D, PAGE)
        owner_t = torch.from_numpy(owner).to(device)
        k_pages, k_scale = _fp8_pool(kshape, gen, device, live[:, None, None, :, None], owner_t, B, H_kv, (2, 3, 4))
        v_pages, v_scale = _fp8_pool(vshape, gen, device, live[:, None, None, :], owner_t, B, H_kv, (2, 3))
        q = _bf16_normal((T, H_q, D), gen, device)
        tok_req = torch.from_numpy(np.repeat(np.arange(B), new).astype(np.int64)).to(device)
        k_new = _fp8_quantise(torch.randn((T, H_kv, D), generator=gen, device=device), k_scale[tok_req][:, :, None])
        v_new = _fp8_quantise(torch.randn((T, H_kv, D), generator=gen, device=device), v_scale[tok_req][:, :, None])
    return PrefillWorkload(
        name=name or "custom", H_q=H_q, H_kv=H_kv, D=D, scale=float(np.float32(1.0 / math.sqrt(D))),
        cached=cached, new=new, num_pages=NP,
        block_table=torch.from_numpy(bt).to(device),
        seq_lens=torch.from_numpy(cached.astype(np.int32)).to(device),
        q_start=torch.from_numpy(q_start).to(device),
        k_pages=k_pages.contiguous(), v_pages=v_pages.contiguous(), q=q, k_new=k_new.contiguous(),
        v_new=v_new.contiguous(), kv=kv, k_scale=k_scale, v_scale=v_scale)
