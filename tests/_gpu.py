"""Helpers of the GPU tests: run steps through the library, move pools to the
host for the oracle, and compare against the oracle."""
from __future__ import annotations

import os

import numpy as np
import torch

import oracle
import paper_2510_15330_amd as bl
from paper_2510_15330_amd import workloads as wl

# (max-abs, rel-L2) against the binary64 oracle: bf16 K/V, and fp8-e4m3fn K/V.
TOL = {"bf16": (1e-2, 2e-3), "fp8": (3e-2, 1e-2)}


def bits16(t: torch.Tensor) -> np.ndarray:
    return t.detach().contiguous().cpu().view(torch.int16).numpy().view(np.uint16)


def codes(t: torch.Tensor) -> np.ndarray:
    return t.detach().contiguous().cpu().view(torch.uint8).numpy()


def host_codes(t: torch.Tensor, kv: str) -> np.ndarray:
    return bits16(t) if kv == "bf16" else codes(t)


def kv_code(kv):
    return oracle.BF16 if kv == "bf16" else oracle.FP8_E4M3FN


def to_device(w: wl.Workload, device="cuda") -> wl.Workload:
    import dataclasses
    f = {}
    for k, v in dataclasses.asdict(w).items():
        f[k] = v.to(device) if isinstance(v, torch.Tensor) else v
    return wl.Workload(**f)


def gpu_step(w: wl.Workload, step: int, out: torch.Tensor, **kw):
    """One decode step: append this step's token, then attend."""
    bl.kv_append(w.k_new[step], w.v_new[step], w.k_pages, w.v_pages, w.block_table, w.seq_lens)
    bl.decode_attention(w.q[step], w.k_pages, w.v_pages, w.block_table, w.seq_lens, w.scale, out,
                        k_scale=w.k_scale, v_scale=w.v_scale, **kw)


def out_f64(out: torch.Tensor) -> np.ndarray:
    return out.detach().float().cpu().double().numpy()


def errors(got: np.ndarray, ref: np.ndarray):
    diff = got - ref
    max_abs = float(np.abs(diff).max()) if diff.size else 0.0
    nrm = float(np.linalg.norm(ref))
    rel = float(np.linalg.norm(diff) / nrm) if nrm > 0 else float(np.linalg.norm(diff))
    return max_abs, rel


# (test, bound kind, max-abs, rel-L2, what) of every comparison, for the
# margins table the session prints at its end (tests/conftest.py)
MARGINS = []


def assert_close(got, ref, kv, what=""):
    ma, rl = errors(got, ref)
    tol_abs, tol_rel = TOL[kv]
    test = os.environ.get("PYTEST_CURRENT_TEST", "?").split(" ")[0]
    MARGINS.append((test, kv, ma, rl, what))
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    assert ma <= tol_abs and rl <= tol_rel, f"{what}: max-abs {ma:.3e} (<= {tol_abs}), rel-L2 {rl:.3e} (<= {tol_rel})"
    return ma, rl


def oracle_full(w: wl.Workload, q_step: int, seq_lens=None) -> np.ndarray:
    """Oracle over the whole (host-copied) pools at the current state."""
    sl = (w.seq_lens if seq_lens is None else seq_lens).cpu().numpy().astype(np.int32)
    return oracle.decode_attention(
        bits16(w.q[q_step]), host_codes(w.k_pages, w.kv), host_codes(w.v_pages, w.kv),
        w.block_table.cpu().numpy(), sl, w.scale, kv_code(w.kv),
        None if w.k_scale is None else w.k_scale.cpu().numpy(),
        None if w.v_scale is None else w.v_scale.cpu().numpy())


def oracle_rows(w: wl.Workload, q_step: int, reqs) -> np.ndarray:
    """Oracle for a subset of requests: gather their pages into a compact pool
    on the device, copy that to the host and remap the block table."""
    reqs = list(reqs)
    sl = w.seq_lens[reqs].cpu().numpy().astype(np.int32)
    bt = w.block_table[reqs].cpu().numpy()
    need = (sl + 15) // 16
    used = [bt[i, :need[i]] for i in range(len(reqs))]
    pages = np.unique(np.concatenate(used)) if used else np.zeros(0, np.int32)
    remap = {int(p): i for i, p in enumerate(pages)}
    bt2 = np.full((len(reqs), max(int(need.max()), 1)), -1, dtype=np.int32)
    for i, u in enumerate(used):
        bt2[i, :len(u)] = [remap[int(p)] for p in u]
    idx = torch.from_numpy(pages.astype(np.int64)).to(w.k_pages.device)
    kp = w.k_pages.index_select(0, idx)
    vp = w.v_pages.index_select(0, idx)
    ks = vs = None
    if w.kv == "fp8":
        ks = w.k_scale[reqs].cpu().numpy()
        vs = w.v_scale[reqs].cpu().numpy()
    return oracle.decode_attention(bits16(w.q[q_step][reqs]), host_codes(kp, w.kv), host_codes(vp, w.kv),
                                   bt2, sl, w.scale, kv_code(w.kv), ks, vs)
