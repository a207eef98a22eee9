"""Shared driver of the GPU parity tests: draw a workload, run it through the C ABI, run the oracle
on the same inputs (all problems and heads, or a sample), and compare."""
from __future__ import annotations

import dataclasses
import sys
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from oracle import evict, profiles
from paper_2609_30738_amd import _lib, api, workloads
from tests import compare


def layer_lambdas(wl: workloads.Workload, problems: Sequence[int]) -> Tuple[np.ndarray, np.ndarray]:
    """Per-problem fp32 coefficients from the oracle's own profile evaluation."""
    l1 = profiles.layer_lambdas(wl.lam1.family, wl.lam1.params, wl.n_layers)
    l2 = profiles.layer_lambdas(wl.lam2.family, wl.lam2.params, wl.n_layers)
    lam1 = np.array([l1[wl.layer_of(p)] for p in problems], dtype=np.float32)
    lam2 = np.array([l2[wl.layer_of(p)] for p in problems], dtype=np.float32)
    return lam1, lam2


@dataclasses.dataclass
class GpuRun:
    wl: workloads.Workload
    problems: List[int]
    packed: workloads.PackedInputs
    lam1: np.ndarray
    lam2: np.ndarray
    budget: int
    cand_mult: int
    keep_tail: int
    host: Dict[str, np.ndarray]
    pool: int = 1
    w_mu: float = 1.0
    sigma_rows: str = "group_mean"
    budgets: Optional[np.ndarray] = None  # per-problem budgets (budget is then the row stride)

    def budget_of(self, j: int) -> int:
        return self.budget if self.budgets is None else int(self.budgets[j])


def run_gpu(wl: workloads.Workload, problems: Optional[Sequence[int]] = None, *, fused: bool = False,
            want_attn: bool = False, cand_mult: int = 4, keep_tail: Optional[int] = None,
            budget: Optional[int] = None, packed: Optional[workloads.PackedInputs] = None,
            pool: int = 1, w_mu: float = 1.0, sigma_rows: str = "group_mean",
            budgets: Optional[Sequence[int]] = None) -> GpuRun:
    import torch
    probs = list(range(wl.n_prob)) if problems is None else list(problems)
    print(f"[gpu case] {wl.name} problems={len(probs)} fused={fused} attn={want_attn} "
          f"cand_mult={cand_mult} keep_tail={keep_tail} pool={pool} w_mu={w_mu} "
          f"sigma_rows={sigma_rows} budgets={None if budgets is None else list(budgets)}",
          flush=True)
    sys.stdout.flush()
    if packed is None:
        packed = workloads.draw_packed(wl, probs)
    lam1, lam2 = layer_lambdas(wl, probs)
    B = wl.budget if budget is None else budget
    bud = None
    if budgets is not None:
        bud = np.asarray(budgets, dtype=np.int32)
        B = max(B, int(bud.max())) if budget is not None else int(bud.max())
    tail = wl.w if keep_tail is None else keep_tail
    inp = api.upload(wl.dtype, wl.h_q, wl.h_kv, wl.d, wl.w, packed.q_win, packed.k, packed.v,
                     packed.lens, packed.tok_off, lam1, lam2)
    out = api.allocate(inp, B, cand_mult, tail, want_candidates=True, want_attn=want_attn)
    api.run_pass(inp, out, B, cand_mult, tail, fused=fused, pool=pool, w_mu=w_mu,
                 sigma_rows=sigma_rows,
                 budgets=None if bud is None else _lib.Budgets(bud, inp.k.device))
    torch.cuda.synchronize()
    host = {name: api.to_host_bits(getattr(out, name)) for name in
            ("row_max", "row_sum", "mu", "sigma", "sel_idx", "sel_score", "cand_idx", "cand_corr",
             "k_out", "v_out")}
    if want_attn:
        host["attn"] = api.to_host_bits(out.attn)
    return GpuRun(wl, probs, packed, lam1, lam2, B, cand_mult, tail, host, pool, w_mu, sigma_rows,
                  bud)


def problem_arrays(run: GpuRun, j: int):
    """Stored inputs of the j-th problem of the run, [h_q,w,d] and [h_kv,L,d]."""
    wl = run.wl
    L = int(run.packed.lens[j])
    off = int(run.packed.tok_off[j]) * wl.h_kv * wl.d
    n = L * wl.h_kv * wl.d
    k = run.packed.k[off:off + n].reshape(wl.h_kv, L, wl.d)
    v = run.packed.v[off:off + n].reshape(wl.h_kv, L, wl.d)
    return run.packed.q_win[j], k, v


def check_problem(run: GpuRun, j: int, heads: Optional[Sequence[int]] = None,
                  check_compaction: bool = True) -> List[compare.SelectionReport]:
    """Compare problem j of a GPU run with the oracle; returns the selection reports."""
    wl = run.wl
    q, k, v = problem_arrays(run, j)
    L = int(run.packed.lens[j])
    heads = list(range(wl.h_kv)) if heads is None else list(heads)
    where = f"{wl.name} p={run.problems[j]}"
    Bp = run.budget_of(j)
    res = evict.evict_problem(q, k, None, wl.dtype, wl.scale, float(run.lam1[j]),
                              float(run.lam2[j]), Bp, run.cand_mult, run.keep_tail,
                              heads=heads, want_attn="attn" in run.host, pool=run.pool,
                              w_mu=run.w_mu, sigma_all_rows=run.sigma_rows == "all_rows")
    H = run.host
    rows = wl.h_q * wl.w
    compare.assert_row_stats(H["row_max"][j * rows:(j + 1) * rows].reshape(wl.h_q, wl.w),
                             H["row_sum"][j * rows:(j + 1) * rows].reshape(wl.h_q, wl.w),
                             res.row_max, res.row_sum, where)
    tok = int(run.packed.tok_off[j])
    mu = H["mu"][tok * wl.h_kv:(tok + L) * wl.h_kv].reshape(wl.h_kv, L)
    sg = H["sigma"][tok * wl.h_kv:(tok + L) * wl.h_kv].reshape(wl.h_kv, L)
    for g in heads:
        compare.assert_mu_sigma(mu[g], sg[g], res.mu[g], res.sigma[g], f"{where} g={g}")
    if "attn" in H:
        a = H["attn"][tok * wl.h_q * wl.w:(tok + L) * wl.h_q * wl.w].reshape(wl.h_q, wl.w, L)
        np.testing.assert_allclose(a, res.attn, rtol=1e-5, atol=1e-12, err_msg=f"{where}: attn")
        assert np.all(a[res.attn == 0] == 0), f"{where}: masked attention must be exactly 0"
    kd = evict.decode(k, wl.dtype)
    reports = []
    B = run.budget
    stride = H["cand_idx"].size // (len(run.problems) * wl.h_kv)
    for g in heads:
        o = (j * wl.h_kv + g)
        assert np.all(H["sel_idx"][o * B + Bp:(o + 1) * B] == -1), f"{where} g={g}: padding"
        assert np.all(H["sel_score"][o * B + Bp:(o + 1) * B] == 0), f"{where} g={g}: padding"
        sel = H["sel_idx"][o * B:o * B + Bp]
        cand = H["cand_idx"][o * stride:(o + 1) * stride]
        hr = res.heads[g]
        rep = compare.check_selection(hr, kd[g], float(run.lam2[j]), sel, cand, f"{where} g={g}")
        reports.append(rep)
        if rep.diverged_at is None and rep.candidates_equal:
            ss = H["sel_score"][o * B:o * B + Bp]
            tol = [compare.score_tol(float(hr.s_tilde[i]), float(run.lam2[j])) for i in sel]
            bad = np.abs(ss - np.asarray(hr.trace.score)) > np.asarray(tol)
            assert not bad.any(), (f"{where} g={g}: sel_score at steps {np.flatnonzero(bad)[:8]}: "
                                   f"{ss[bad][:4]} vs {np.asarray(hr.trace.score)[bad][:4]}")
            corr = H["cand_corr"][o * stride:o * stride + len(hr.candidates)]
            ref = np.array([float(hr.trace.corr[c]) for c in hr.candidates])
            np.testing.assert_allclose(corr, ref, rtol=1e-5, atol=compare.CORR_ATOL,
                                       err_msg=f"{where} g={g}: corr")
            assert np.all(cand[len(hr.candidates):] == -1)
        if check_compaction and rep.diverged_at is None and rep.candidates_equal:
            # same admissions as the oracle: the compacted rows must be the oracle's, byte for byte
            rows_out = Bp + run.keep_tail  # rows written; the block's stride is B + keep_tail
            keep = evict.kept_positions(hr.trace.selected, L, run.keep_tail)
            base = o * (B + run.keep_tail) * wl.d
            ko = H["k_out"][base:base + rows_out * wl.d].reshape(rows_out, wl.d)
            vo = H["v_out"][base:base + rows_out * wl.d].reshape(rows_out, wl.d)
            np.testing.assert_array_equal(ko, evict.compact_rows(k[g], keep),
                                          err_msg=f"{where} g={g}: compacted K")
            np.testing.assert_array_equal(vo, evict.compact_rows(v[g], keep),
                                          err_msg=f"{where} g={g}: compacted V")
    return reports


def summarize(reports: List[compare.SelectionReport]) -> str:
    steps = sum(r.steps for r in reports)
    exact = sum(r.exact_steps for r in reports)
    div = [r for r in reports if r.diverged_at is not None]
    near = sum(r.near_ties for r in reports)
    cert = sum(1 for r in reports if r.near_ties == 0)
    worst = max((r.divergence_margin for r in div if r.divergence_margin is not None),
                default=None)
    return (f"heads={len(reports)} fully-certified-heads={cert} steps={steps} "
            f"identical-to-oracle={exact} near-ties(oracle)={near} diverged-heads={len(div)}"
            + (f" largest-relative-margin-at-divergence={worst:.2g}" if worst is not None else ""))
