"""Device plumbing around the C ABI: upload inputs, allocate outputs, run one eviction pass.

Torch is used only for device memory and streams; every step of the pass is one of the library's
entry points (kv_window_scores + kv_mu_sigma or kv_window_mu_sigma, kv_mmr_select or
kv_mmr_select_ex, kv_compact_cache or kv_compact_cache_ex), or their _ex variants.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

from . import _lib


def to_device(arr: np.ndarray, device="cuda"):
    """Upload a host array; uint16 arrays are bf16 bit patterns and become torch.bfloat16."""
    import torch
    if arr.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).to(device).view(
            torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(arr)).to(device)


def to_host_bits(t) -> np.ndarray:
    """Download a device tensor; bf16 comes back as uint16 bit patterns."""
    import torch
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


@dataclasses.dataclass
class DeviceInputs:
    batch: _lib.Batch
    q_win: object
    k: object
    v: object
    lambda1: object
    lambda2: object
    scale: float


def upload(dtype: str, h_q: int, h_kv: int, d: int, w: int, q_win: np.ndarray, k: np.ndarray,
           v: np.ndarray, lens: np.ndarray, tok_off: np.ndarray, lambda1: np.ndarray,
           lambda2: np.ndarray, scale: Optional[float] = None, device="cuda") -> DeviceInputs:
    batch = _lib.Batch(dtype, h_q, h_kv, d, w, lens, tok_off, device=device)
    return DeviceInputs(batch, to_device(q_win, device), to_device(k, device),
                        to_device(v, device),
                        to_device(np.asarray(lambda1, dtype=np.float32), device),
                        to_device(np.asarray(lambda2, dtype=np.float32), device),
                        float(1.0 / np.sqrt(d)) if scale is None else float(scale))


@dataclasses.dataclass
class PassOutputs:
    row_max: object
    row_sum: object
    mu: object
    sigma: object
    sel_idx: object
    sel_score: Optional[object]
    cand_idx: Optional[object]
    cand_corr: Optional[object]
    k_out: object
    v_out: object
    ws: object
    attn: Optional[object] = None


def allocate(inp: DeviceInputs, budget: int, cand_mult: int = 4, keep_tail: Optional[int] = None,
             want_candidates: bool = False, want_attn: bool = False) -> PassOutputs:
    import torch
    b = inp.batch
    dev = inp.k.device
    tail = b.w if keep_tail is None else keep_tail
    n_rows = b.n_prob * b.h_q * b.w
    tokens = b.total_tokens
    ws_bytes = _lib.workspace_bytes(b, budget, cand_mult, tail)
    f32 = dict(dtype=torch.float32, device=dev)
    stride = _lib.candidate_stride(b, budget, cand_mult, tail) if want_candidates else 0
    return PassOutputs(
        row_max=torch.empty(n_rows, **f32), row_sum=torch.empty(n_rows, **f32),
        mu=torch.empty(tokens * b.h_kv, **f32), sigma=torch.empty(tokens * b.h_kv, **f32),
        sel_idx=torch.empty(b.n_prob * b.h_kv * budget, dtype=torch.int32, device=dev),
        sel_score=torch.empty(b.n_prob * b.h_kv * budget, **f32) if want_candidates else None,
        cand_idx=(torch.empty(b.n_prob * b.h_kv * stride, dtype=torch.int32, device=dev)
                  if want_candidates else None),
        cand_corr=torch.empty(b.n_prob * b.h_kv * stride, **f32) if want_candidates else None,
        k_out=torch.empty(b.n_prob * b.h_kv * (budget + tail) * b.d, dtype=inp.k.dtype,
                          device=dev),
        v_out=torch.empty(b.n_prob * b.h_kv * (budget + tail) * b.d, dtype=inp.v.dtype,
                          device=dev),
        ws=torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device=dev),
        attn=torch.empty(tokens * b.h_q * b.w, **f32) if want_attn else None)


def run_pass(inp: DeviceInputs, out: PassOutputs, budget: int, cand_mult: int = 4,
             keep_tail: Optional[int] = None, fused: bool = True, pool: int = 1, w_mu: float = 1.0,
             sigma_rows: str = "group_mean", budgets: Optional[_lib.Budgets] = None,
             stream=None) -> None:
    """One whole eviction pass over the batch, enqueued on `stream` (default: current stream).

    pool / w_mu: scoring options of kv_mmr_select_ex (max-pool window, weight of mu);
    sigma_rows: the dispersion reading of kv_mu_sigma_ex / kv_window_mu_sigma_ex; budgets:
    per-problem budgets (then `budget` is the row stride and must be at least their maximum).  The
    defaults call the plain entry points."""
    b = inp.batch
    tail = b.w if keep_tail is None else keep_tail
    plain = sigma_rows == "group_mean"
    if fused and out.attn is None:
        if plain:
            _lib.window_mu_sigma(b, inp.q_win, inp.k, inp.scale, out.row_max, out.row_sum, out.mu,
                                 out.sigma, out.ws, stream)
        else:
            _lib.window_mu_sigma_ex(b, inp.q_win, inp.k, inp.scale, sigma_rows, out.row_max,
                                    out.row_sum, out.mu, out.sigma, out.ws, stream)
    else:
        _lib.window_scores(b, inp.q_win, inp.k, inp.scale, out.row_max, out.row_sum, out.ws,
                           stream)
        if plain:
            _lib.mu_sigma(b, inp.q_win, inp.k, inp.scale, out.row_max, out.row_sum, out.mu,
                          out.sigma, out.attn, stream)
        else:
            _lib.mu_sigma_ex(b, inp.q_win, inp.k, inp.scale, out.row_max, out.row_sum, sigma_rows,
                             out.mu, out.sigma, out.attn, stream)
    if pool == 1 and w_mu == 1.0 and budgets is None:
        _lib.mmr_select(b, out.mu, out.sigma, inp.k, inp.lambda1, inp.lambda2, budget, cand_mult,
                        tail, out.sel_idx, out.sel_score, out.cand_idx, out.cand_corr, out.ws,
                        stream)
        _lib.compact_cache(b, inp.k, inp.v, out.sel_idx, budget, tail, out.k_out, out.v_out,
                           stream)
    else:
        _lib.mmr_select_ex(b, out.mu, out.sigma, inp.k, inp.lambda1, inp.lambda2, budget,
                           cand_mult, tail, out.sel_idx, out.sel_score, out.cand_idx,
                           out.cand_corr, out.ws, pool=pool, w_mu=w_mu, budgets=budgets,
                           stream=stream)
        _lib.compact_cache_ex(b, inp.k, inp.v, out.sel_idx, budget, tail, budgets, out.k_out,
                              out.v_out, stream=stream)
