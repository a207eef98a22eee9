"""Comparison of GPU results with the CPU oracle.

Statistics (row max/sum, attention, mu, sigma) are compared element by element within the fp32
tolerances below; every candidate's corr and every step's score are compared with the oracle's
values for the same admission history.

Selections are integer results decided by fp32 arithmetic (R23).  Per kv head:
  * the candidate set (top C of s, section 3.2): identical to the oracle's where the oracle's margin
    at the cut is certified (tests/certify.py); otherwise (a cut through the flat bulk of the
    scores) the sets may differ only by tokens whose base scores lie within the fp32 error of the
    cut value, which is checked;
  * the greedy admissions (Eq. (5)): the oracle's greedy is run on the GPU's candidate set (the
    oracle's own trace when the sets are equal) and its margins certified; a certified greedy
    must be reproduced exactly, in admission order (with lambda2 = 0, where only the set is
    decided, the set exactly and the order step by step within the score tolerance).  An
    uncertified greedy is replayed: each admitted position must be an argmax of s~ + lambda2 corr
    within the score tolerance, given the GPU's own earlier admissions;
  * sel_score and cand_corr are compared with the oracle's values for the GPU's own admission
    sequence, and the compacted rows with the rows at the GPU's own selection, byte for byte.
"""
from __future__ import annotations

import dataclasses
from fractions import Fraction
from typing import List, Optional, Sequence

import numpy as np

from oracle import evict
from tests import certify

# fp32 error model of the GPU path (the comparator of the scope table: 1e-5 relative in fp32):
# mu to 1e-5 relative; sigma to 1e-5 relative plus 1e-6 mu, since sigma is formed from values of
# size mu and fp32 rounding of those values alone moves sigma by ~1e-6 mu; corr to 1e-5 relative
# plus 1e-6 absolute.  A per-step score s~ + lambda2 corr is a sum of two terms with their own
# errors: s~ = s / max s is a ratio of two base scores, each within 1e-5 of its value, hence within
# 2e-5 |s~|, and lambda2 corr within |lambda2| (1e-5 |corr| + 1e-6); the bound is taken on the terms
# (the score itself can be far smaller than either where they cancel), plus 1e-6 for its rounding.
MU_RTOL = 1e-5
SIGMA_RTOL = 1e-5
SIGMA_MU_FLOOR = 1e-6
STAT_ATOL_FRAC = 1e-12   # of the largest mean in the head
CORR_RTOL = 1e-5
CORR_ATOL = 1e-6
SCORE_RTOL = 2e-5        # of |s~|
SCORE_ATOL = 1e-6
BOUNDARY_RTOL = 2e-5     # relative error of a base score at a cut through the bulk
# replay of an uncertified greedy: two candidates' scores may swap within the sum of their errors
PAIR_RTOL = 2e-5
PAIR_PER_LAMBDA = 4e-6


def order_key(x: np.ndarray) -> np.ndarray:
    """Order-preserving uint32 key of fp32 values (larger value, larger key), as the kernels form it:
    the complemented word for a set sign bit, else the word with the sign bit set."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    return np.where(u & np.uint32(0x80000000), ~u, u | np.uint32(0x80000000))


def _round_f32_exact(x: Fraction) -> np.float32:
    """The fp32 value nearest to the rational x, ties to an even significand."""
    r = np.float32(float(x))
    best, best_d = None, None
    for c in (np.nextafter(r, np.float32(-np.inf)), r, np.nextafter(r, np.float32(np.inf))):
        if not np.isfinite(c):
            continue
        d = abs(Fraction(float(c)) - x)
        if best is None or d < best_d or (d == best_d and int(c.view(np.uint32)) % 2 == 0):
            best, best_d = c, d
    return best


def assert_fma_f32(got: np.ndarray, a: float, b: np.ndarray, c: np.ndarray, where: str) -> None:
    """got == fp32(a * b + c) with one rounding, bit for bit (a, b, c fp32).  The exact product of
    two fp32 values fits a float64, so a float64 sum rounded to fp32 is the fused result except
    where the sum itself rounds next to an fp32 rounding boundary; every element where that
    evaluation disagrees is decided in exact rational arithmetic."""
    a32 = np.float32(a)
    b32 = np.asarray(b, dtype=np.float32)
    c32 = np.asarray(c, dtype=np.float32)
    got = np.asarray(got, dtype=np.float32)
    fin = np.isfinite(b32) & np.isfinite(c32)
    with np.errstate(over="ignore", invalid="ignore"):
        approx = (np.float64(a32) * b32.astype(np.float64) + c32.astype(np.float64)).astype(np.float32)
    same = (got.view(np.uint32) == approx.view(np.uint32)) | (np.isnan(got) & np.isnan(approx))
    for i in np.flatnonzero(~same & fin):
        want = _round_f32_exact(Fraction(float(a32)) * Fraction(float(b32[i])) + Fraction(float(c32[i])))
        assert got[i].view(np.uint32) == want.view(np.uint32), (
            f"{where}[{i}]: {got[i]!r} is not fma({a32!r}, {b32[i]!r}, {c32[i]!r}) = {want!r}")
    bad = ~same & ~fin
    assert not bad.any(), f"{where}: non-finite inputs give {got[bad][:4]} instead of {approx[bad][:4]}"


def pair_tol(st_a: float, st_b: float, lam2: float) -> float:
    """How far apart the fp32 scores s~ + lambda2 corr of two candidates may be and still swap."""
    return PAIR_RTOL * (abs(st_a) + abs(st_b)) + PAIR_PER_LAMBDA * abs(lam2)


@dataclasses.dataclass
class ErrStats:
    """Largest observed errors: mu and sigma relative (sigma where sigma > 1e-3 mu), corr
    absolute, per-step score as a fraction of its tolerance."""
    mu_rel: float = 0.0
    sigma_rel: float = 0.0
    corr_abs: float = 0.0
    score_tol_frac: float = 0.0

    def merge(self, o: "ErrStats") -> None:
        for f in dataclasses.fields(self):
            setattr(self, f.name, max(getattr(self, f.name), getattr(o, f.name)))

    def text(self) -> str:
        return (f"max-err mu={self.mu_rel:.2g}rel sigma={self.sigma_rel:.2g}rel "
                f"corr={self.corr_abs:.2g}abs score={self.score_tol_frac:.2g}xtol")


def assert_mu_sigma(mu: np.ndarray, sigma: np.ndarray, ref_mu: np.ndarray, ref_sigma: np.ndarray,
                    where: str, err: Optional[ErrStats] = None) -> None:
    floor = STAT_ATOL_FRAC * float(ref_mu.max())
    mu_err = np.abs(mu - ref_mu)
    bad = mu_err > MU_RTOL * np.abs(ref_mu) + floor
    assert not bad.any(), (f"{where}: mu mismatch at {np.flatnonzero(bad)[:8]} "
                           f"gpu {mu[bad][:4]} ref {ref_mu[bad][:4]}")
    sg_err = np.abs(sigma - ref_sigma)
    bad = sg_err > SIGMA_RTOL * np.abs(ref_sigma) + SIGMA_MU_FLOOR * np.abs(ref_mu) + floor
    assert not bad.any(), (f"{where}: sigma mismatch at {np.flatnonzero(bad)[:8]} "
                           f"gpu {sigma[bad][:4]} ref {ref_sigma[bad][:4]}")
    if err is not None:
        nz = ref_mu > 0
        if nz.any():
            err.mu_rel = max(err.mu_rel, float((mu_err[nz] / ref_mu[nz]).max()))
        nz = ref_sigma > 1e-3 * ref_mu
        if nz.any():
            err.sigma_rel = max(err.sigma_rel, float((sg_err[nz] / ref_sigma[nz]).max()))


def assert_row_stats(row_max, row_sum, ref_max, ref_sum, where: str) -> None:
    np.testing.assert_allclose(row_max, ref_max, rtol=1e-5, atol=1e-5, err_msg=f"{where}: row_max")
    np.testing.assert_allclose(row_sum, ref_sum, rtol=1e-5, err_msg=f"{where}: row_sum")


@dataclasses.dataclass
class SelectionReport:
    steps: int
    identical_steps: int        # steps identical to the reference trace before any divergence
    certified: bool             # the oracle certified both the cut and the greedy (stored inputs)
    candidates_equal: bool
    set_equal: bool             # admitted set identical to the oracle's
    greedy_certified: bool      # the reference greedy (on the GPU's candidates) is certified
    boundary: str
    err: ErrStats = dataclasses.field(default_factory=ErrStats)


@dataclasses.dataclass
class Replay:
    scores: List[float]  # the oracle's fp32 score of each GPU admission, given the GPU's history
    corr: dict           # each candidate's corr when admitted, else after the last step


def replay(h: evict.HeadResult, k_unit: np.ndarray, cand: Sequence[int], lam2: float,
           sel: Sequence[int], check_from: Optional[int], where: str) -> Replay:
    """The oracle's scores along the GPU's admission sequence; from step check_from on (None: no
    check) every admission must be an argmax within the pair tolerance."""
    lam = float(np.float32(lam2))
    cand = np.asarray(sorted(cand))
    pos = {int(c): j for j, c in enumerate(cand)}
    s_t = np.array([h.s_tilde[c] for c in cand], dtype=np.float64)
    corr = np.zeros(len(cand), dtype=np.float32)
    taken = np.zeros(len(cand), dtype=bool)
    out_scores = []
    corr_at = {}
    for t, j in enumerate(sel):
        j = int(j)
        assert j in pos, f"{where}: step {t} admitted {j}, not a candidate"
        jj = pos[j]
        assert not taken[jj], f"{where}: step {t} admitted {j} twice"
        score = (s_t + lam * corr.astype(np.float64)).astype(np.float32).astype(np.float64)
        out_scores.append(float(score[jj]))
        corr_at[j] = float(corr[jj])
        if check_from is not None and t >= check_from:
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
    for c, j in pos.items():
        if c not in corr_at:
            corr_at[c] = float(corr[j])
    return Replay(out_scores, corr_at)


def check_candidates(h: evict.HeadResult, cand: Sequence[int], where: str) -> bool:
    """GPU candidate positions against the oracle's; returns whether they are equal (a difference is
    allowed only among near-ties at the cut)."""
    assert len(cand) == len(h.candidates), f"{where}: candidate count {len(cand)}"
    if list(cand) == list(h.candidates):
        return True
    assert h.boundary_gap is not None, f"{where}: candidate sets differ without a cut"
    s_c = h.boundary_gap[0]
    for i in set(cand) ^ set(h.candidates):
        assert abs(float(h.s[i]) - s_c) <= BOUNDARY_RTOL * abs(s_c), (
            f"{where}: candidate {i} (s={h.s[i]:.9g}) differs away from the cut {s_c:.9g}")
    return False


def check_selection(h: evict.HeadResult, k_head: np.ndarray, lam2: float, sel: Sequence[int],
                    cand: Sequence[int], budget: int, certified: bool, dtype: str,
                    sel_score: Optional[np.ndarray] = None, cand_corr: Optional[np.ndarray] = None,
                    where: str = "") -> SelectionReport:
    """One head's GPU selection against the oracle (see the module docstring).

    k_head: the head's stored keys [L, d]; cand: the GPU's candidate positions (ascending);
    certified: the oracle certified this head's cut and greedy on these inputs, so the GPU must
    reproduce the oracle exactly.  sel_score / cand_corr (optional): the GPU's outputs for them."""
    sel = [int(x) for x in sel]
    cand = [int(c) for c in cand]
    cand_equal = check_candidates(h, cand, where)
    if certified:
        assert cand_equal, f"{where}: certified head, candidate set differs from the oracle's"
    kd = evict.decode(k_head, dtype)
    k_unit = np.zeros_like(kd)
    k_unit[cand] = evict.unit_keys(kd[cand])
    if cand_equal:
        ref = h.trace
    else:
        ref = evict.greedy_mmr(h.s_tilde, k_unit, cand, lam2, budget)
    g_stat, _, _, _ = certify.certify_greedy(h, k_head, lam2, dtype, ref, cand)
    g_cert = g_stat == "certified"
    lam0 = float(np.float32(lam2)) == 0.0
    if certified:
        assert g_cert, f"{where}: certified head, greedy margins not certified"
    div = next((t for t, (a, b) in enumerate(zip(sel, ref.selected)) if a != b), None)
    if g_cert and not lam0:
        assert div is None and len(sel) == len(ref.selected), (
            f"{where}: certified greedy, GPU admits {sel[div] if div is not None else sel} at step "
            f"{div}, oracle {ref.selected[div] if div is not None else ref.selected}")
    if g_cert and lam0:
        assert set(sel) == set(ref.selected), f"{where}: certified set differs"
    check_from = None if (g_cert and not lam0) else 0
    rp = replay(h, k_unit, cand, lam2, sel, check_from, where)
    err = ErrStats()
    if sel_score is not None:
        ref_sc = np.asarray(rp.scores)
        d = np.abs(np.asarray(sel_score, dtype=np.float64) - ref_sc)
        st_sel = np.array([abs(float(h.s_tilde[j])) for j in sel])
        corr_sel = np.array([abs(rp.corr[j]) for j in sel])
        lam = abs(float(np.float32(lam2)))
        tol = SCORE_RTOL * st_sel + lam * (CORR_RTOL * corr_sel + CORR_ATOL) + SCORE_ATOL
        bad = d > tol
        assert not bad.any(), (f"{where}: sel_score at steps {np.flatnonzero(bad)[:8]}: "
                               f"{np.asarray(sel_score)[bad][:4]} vs {ref_sc[bad][:4]}")
        if d.size:
            err.score_tol_frac = float((d / tol).max())
    if cand_corr is not None:
        ref_c = np.array([rp.corr[c] for c in cand])
        d = np.abs(np.asarray(cand_corr, dtype=np.float64) - ref_c)
        bad = d > CORR_RTOL * np.abs(ref_c) + CORR_ATOL
        assert not bad.any(), (f"{where}: cand_corr at {np.flatnonzero(bad)[:8]}: "
                               f"{np.asarray(cand_corr)[bad][:4]} vs {ref_c[bad][:4]}")
        err.corr_abs = float(d.max()) if d.size else 0.0
    return SelectionReport(len(sel), div if div is not None else len(sel), certified, cand_equal,
                           set(sel) == set(h.trace.selected), g_cert, "", err)


def summarize(reports: List[SelectionReport]) -> str:
    steps = sum(r.steps for r in reports)
    ident = sum(r.identical_steps for r in reports)
    err = ErrStats()
    for r in reports:
        err.merge(r.err)
    return (f"heads={len(reports)} certified-heads={sum(r.certified for r in reports)} "
            f"identical-candidate-sets={sum(r.candidates_equal for r in reports)} "
            f"identical-selected-sets={sum(r.set_equal for r in reports)} "
            f"greedy-certified={sum(r.greedy_certified for r in reports)} "
            f"steps={steps} identical-to-reference={ident} | {err.text()}")
