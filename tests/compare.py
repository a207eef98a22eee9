"""Comparison of GPU results with the CPU oracle.

Statistics (row max/sum, attention, mu, sigma, corr) are compared element by element within the
fp32 tolerances below.  Selections are integer results decided by fp32 arithmetic: where the
oracle's decision has a clear margin over its runner-up the GPU must make the same decision; at a
near-tie (margin within the fp32 error of the scores) several answers are correct, so the GPU's
choice and every later step are checked for validity instead: each admitted position must be an
(approximate) argmax of s~ + lambda2 corr given the positions admitted before it, recomputed by
the oracle's own functions.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Sequence

import numpy as np

from oracle import evict

# fp32 error model of the GPU path: statistics within 1e-5 relative (sigma with a floor of
# 1e-6 mu, since sigma is formed from values of size mu), cosines within 2e-6 absolute, and the
# scores built from them within the sum of their parts.
MU_RTOL = 1e-5
SIGMA_RTOL = 1e-5
SIGMA_MU_FLOOR = 1e-6
STAT_ATOL_FRAC = 1e-12   # of the largest mean in the head
CORR_ATOL = 2e-6
SCORE_RTOL = 2e-5        # relative error of s~ (mu and sigma to 1e-5, plus the normaliser)
SCORE_PER_LAMBDA = 2 * CORR_ATOL  # error of lambda2 * corr per unit |lambda2|
BOUNDARY_RTOL = 2e-5     # relative error of a base score


def pair_tol(st_a: float, st_b: float, lam2: float) -> float:
    """How far apart the fp32 scores s~ + lambda2 corr of two candidates may be and still swap."""
    return SCORE_RTOL * (abs(st_a) + abs(st_b)) + SCORE_PER_LAMBDA * abs(lam2)


def score_tol(st: float, lam2: float) -> float:
    """Error bound of one candidate's score."""
    return SCORE_RTOL * abs(st) + 0.5 * SCORE_PER_LAMBDA * abs(lam2)


def assert_mu_sigma(mu: np.ndarray, sigma: np.ndarray, ref_mu: np.ndarray, ref_sigma: np.ndarray,
                    where: str) -> None:
    floor = STAT_ATOL_FRAC * float(ref_mu.max())
    mu_err = np.abs(mu - ref_mu)
    bad = mu_err > MU_RTOL * np.abs(ref_mu) + floor
    assert not bad.any(), (f"{where}: mu mismatch at {np.flatnonzero(bad)[:8]} "
                           f"gpu {mu[bad][:4]} ref {ref_mu[bad][:4]}")
    sg_err = np.abs(sigma - ref_sigma)
    bad = sg_err > SIGMA_RTOL * np.abs(ref_sigma) + SIGMA_MU_FLOOR * np.abs(ref_mu) + floor
    assert not bad.any(), (f"{where}: sigma mismatch at {np.flatnonzero(bad)[:8]} "
                           f"gpu {sigma[bad][:4]} ref {ref_sigma[bad][:4]}")


def assert_row_stats(row_max, row_sum, ref_max, ref_sum, where: str) -> None:
    np.testing.assert_allclose(row_max, ref_max, rtol=1e-5, atol=1e-5, err_msg=f"{where}: row_max")
    np.testing.assert_allclose(row_sum, ref_sum, rtol=1e-5, err_msg=f"{where}: row_sum")


@dataclasses.dataclass
class SelectionReport:
    steps: int
    exact_steps: int           # steps identical to the oracle before any divergence
    near_ties: int             # oracle steps whose margin is within the score tolerance
    diverged_at: Optional[int]
    candidates_equal: bool
    divergence_margin: Optional[float] = None  # oracle margin at the divergence, relative to s~


def _valid_replay(h: evict.HeadResult, k_unit: np.ndarray, cand: Sequence[int], lam2: float,
                  sel: Sequence[int], start: int, where: str) -> None:
    """Check sel[start:] step by step against the oracle's scores given sel[:t]."""
    lam = float(np.float32(lam2))
    cand = np.asarray(sorted(cand))
    pos = {int(c): j for j, c in enumerate(cand)}
    s_t = np.array([h.s_tilde[c] for c in cand], dtype=np.float64)
    corr = np.zeros(len(cand), dtype=np.float32)
    taken = np.zeros(len(cand), dtype=bool)
    for t, j in enumerate(sel):
        j = int(j)
        assert j in pos, f"{where}: step {t} admitted {j}, not a candidate"
        jj = pos[j]
        assert not taken[jj], f"{where}: step {t} admitted {j} twice"
        if t >= start:
            score = (s_t + lam * corr.astype(np.float64)).astype(np.float32).astype(np.float64)
            score[taken] = -np.inf
            bi = int(np.argmax(score))
            tol = pair_tol(s_t[jj], s_t[bi], lam2)
            assert score[jj] >= score[bi] - tol, (
                f"{where}: step {t} admitted {j} with score {score[jj]:.9g}, best "
                f"{score[bi]:.9g} at {int(cand[bi])} (tol {tol:.2g})")
        taken[jj] = True
        cos = (k_unit[cand] @ k_unit[j]).astype(np.float32)
        upd = ~taken & (cos > corr)
        corr[upd] = cos[upd]


def check_selection(h: evict.HeadResult, k_head: np.ndarray, lam2: float, sel: Sequence[int],
                    cand: Optional[Sequence[int]] = None, where: str = "") -> SelectionReport:
    """Compare one head's GPU admissions (admission order) with the oracle's HeadResult.

    k_head: the head's keys in float64 [L, d].  cand: GPU candidate positions (optional).
    """
    sel = [int(x) for x in sel]
    ora = h.trace.selected
    margins = [a - b for a, b in zip(h.trace.score, h.trace.runner_up_score)]
    tols = [pair_tol(h.s_tilde[a], h.s_tilde[b] if b is not None else 0.0, lam2)
            for a, b in zip(ora, h.trace.runner_up)]
    near = sum(1 for m, tl in zip(margins, tols) if m <= tl)
    cand_equal = True
    use_cand = h.candidates
    if cand is not None:
        cand = sorted(int(c) for c in cand if c >= 0)
        assert len(cand) == len(h.candidates), f"{where}: candidate count {len(cand)}"
        if cand != h.candidates:
            cand_equal = False
            # differences are only allowed among near-tied scores at the top-C boundary
            assert h.boundary_gap is not None, f"{where}: candidate sets differ without a boundary"
            s_c = h.boundary_gap[0]
            diff = set(cand) ^ set(h.candidates)
            for i in diff:
                assert abs(float(h.s[i]) - s_c) <= BOUNDARY_RTOL * abs(s_c), (
                    f"{where}: candidate {i} (s={h.s[i]:.9g}) differs away from the boundary "
                    f"{s_c:.9g}")
            use_cand = cand
    div = next((t for t, (a, b) in enumerate(zip(sel, ora)) if a != b), None)
    if div is None and cand_equal:
        assert len(sel) == len(ora)
        return SelectionReport(len(sel), len(sel), near, None, True)
    start = 0 if not cand_equal else div
    rel = None
    if cand_equal:
        assert margins[div] <= tols[div], (
            f"{where}: step {div} admitted {sel[div]} but the oracle admits {ora[div]} by a margin "
            f"{margins[div]:.3g} > {tols[div]:.3g}")
        rel = margins[div] / max(abs(float(h.s_tilde[ora[div]])), 1e-30)
    k_unit = np.zeros_like(k_head)
    k_unit[use_cand] = evict.unit_keys(k_head[use_cand])
    _valid_replay(h, k_unit, use_cand, lam2, sel, start, where)
    return SelectionReport(len(sel), div if div is not None else len(sel), near, div, cand_equal,
                           rel)
