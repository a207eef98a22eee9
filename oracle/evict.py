"""Plain CPU oracle of the post-prefill eviction-scoring path (sections 3.1 and 3.2).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Everything numerical is float64, computed from the exact values of the stored inputs (fp32, or bf16
decoded exactly).  The paper fixes no precision for the selection, so the integer decisions it makes
(the top-4B candidate restriction and every greedy argmax) are taken in fp32, the precision of the
GPU kernels: the statistics are computed in float64, rounded once to fp32, and the decision
quantities are formed in fp32 with one rounding per operation (a multiply-add rounds once).
Besides each decision the oracle records the runner-up, so a comparison can tell a decision that is
fixed by a clear margin from a near-tie where several answers are correct.

Readings of points the paper leaves open (each used below where it applies):
  R1  grouped-query attention: the G query heads that share a kv head are averaged,
      a[r, i] = mean_h A[h, r, i]; the mean (Eq. (1)) and the sample standard deviation (Eq. (3)) are
      then taken over the W window rows, and selection is per kv head.  The other reading (R1b,
      all_rows=True below) takes the mean and the sample standard deviation over all G W
      (head, row) attention values of the group; the mean is the same under both readings.
  R2  causal mask: window row r sits at position L - W + r and attends to keys 0 .. L - W + r.
  R3  the softmax scale is an explicit argument (1/sqrt(d) for scaled dot-product attention).
  R4  candidates are the positions [0, L - keep_tail); the last keep_tail positions (the window by
      default) are always kept.
  R5  the budget B counts greedy admissions; the compacted cache holds B + keep_tail rows.
  R7  the normaliser max_j s_j is clamped below at 1e-12.
  R8  the normaliser's maximum runs over all candidates.
  R9  the top-4B restriction is part of the method (cand_mult = 4); cand_mult = 0 runs the greedy over
      all candidates.
  R10 ties go to the lower position, both at the top-4B boundary and in every argmax.
  R11 corr(i, S) = max(0, max_{j in S} cos) is kept as a running maximum that starts at 0.
  R12 a zero key has a zero unit vector (its cosine to anything is 0).
  R14 selections are reported in admission order; the compacted cache holds the kept positions in
      ascending order followed by the kept tail.

Parity unpinned: R1 (how the query heads of a group enter mu and sigma; token_statistics) and R6
(the size and placement of max_pool) are readings the paper does not fix.  The tests pin both
functions to their own definitions (library mean / stdev, scipy's maximum filter), not to the
paper.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional

import numpy as np

NORMALISER_FLOOR = 1e-12  # R7


# ------------------------------------------------------------------------------------------------
# Inputs
# ------------------------------------------------------------------------------------------------

def decode(x: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 values of stored inputs: fp32 arrays, or bf16 given as uint16 bit patterns."""
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32).astype(np.float64)
    if dtype == "bf16":
        bits = np.asarray(x, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return bits.view(np.float32).astype(np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")


# ------------------------------------------------------------------------------------------------
# Section 3.1: observation-window attention
# ------------------------------------------------------------------------------------------------

def window_logits(q_win: np.ndarray, k: np.ndarray, scale: float) -> np.ndarray:
    """Scaled logits of the W window queries against all L keys, -inf where masked (R2, R3).

    q_win [h_q, W, d] and k [h_kv, L, d] in float64; query head h reads kv head h // (h_q / h_kv).
    Returns l [h_q, W, L].
    """
    h_q, w, _ = q_win.shape
    h_kv, L, _ = k.shape
    group = h_q // h_kv
    logits = np.empty((h_q, w, L), dtype=np.float64)
    for h in range(h_q):
        logits[h] = scale * (q_win[h] @ k[h // group].T)
    for r in range(w):
        logits[:, r, L - w + r + 1:] = -np.inf
    return logits


def window_row_stats(logits: np.ndarray):
    """Per window row: the maximum logit m and the normaliser Z = sum_i exp(l_i - m)."""
    m = logits.max(axis=-1)
    z = np.exp(logits - m[..., None]).sum(axis=-1)
    return m, z


def window_attention(logits: np.ndarray) -> np.ndarray:
    """A[h, r, i] = exp(l - m) / Z: the attention token i receives from window query r (section 3.1)."""
    m, z = window_row_stats(logits)
    return np.exp(logits - m[..., None]) / z[..., None]


def token_statistics(attn: np.ndarray, h_kv: int, all_rows: bool = False):
    """Mean mu_i (Eq. (1)) and sample dispersion sigma_i (Eq. (3)) per kv head, following R1
    (all_rows=False) or R1b (all_rows=True).

    attn [h_q, W, L] -> mu, sigma [h_kv, L].  sigma divides by n - 1 (n = W, or G W under R1b) and
    is computed in two passes (mean first, then the squared deviations from it).
    """
    h_q, w, L = attn.shape
    group = h_q // h_kv
    if all_rows:
        x = attn.reshape(h_kv, group * w, L)
        n = group * w
        mu = x.sum(axis=1) / n
        dev = x - mu[:, None, :]
        return mu, np.sqrt((dev * dev).sum(axis=1) / (n - 1))
    a = attn.reshape(h_kv, group, w, L).sum(axis=1) / group
    mu = a.sum(axis=1) / w
    dev = a - mu[:, None, :]
    sigma = np.sqrt((dev * dev).sum(axis=1) / (w - 1))
    return mu, sigma


# ------------------------------------------------------------------------------------------------
# Section 3.2: base score, normalisation, top-4B restriction, greedy MMR admission
# ------------------------------------------------------------------------------------------------

def f32(x):
    return np.float32(x)


def base_scores(mu: np.ndarray, sigma: np.ndarray, lam1: float, w_mu: float = 1.0) -> np.ndarray:
    """s_i = w_mu mu_i + lambda1 sigma_i (Eq. (2) without the set term), formed in fp32: the weighted
    mean rounded to fp32, then one rounding of the sum.  w_mu = 1 is the paper's score; w_mu = 0
    drops the mean (the "dispersion & Corr" rule of the term ablation, section 4)."""
    mu32 = mu.astype(np.float32)
    if w_mu != 1.0:
        mu32 = (mu32.astype(np.float64) * float(f32(w_mu))).astype(np.float32)
    sg32 = sigma.astype(np.float32).astype(np.float64)
    lam = float(f32(lam1))
    return (mu32.astype(np.float64) + lam * sg32).astype(np.float32)


def max_pool(s: np.ndarray, n_cand: int, pool: int) -> np.ndarray:
    """Max-pooling of the base scores along the candidate positions (the pooling of the mean-attention
    baselines that section 3.1 keeps): s'_i = max of s_j over |j - i| <= (pool - 1) / 2 and
    0 <= j < n_cand, i.e. positions outside the candidate range count as -inf.  pool is odd."""
    if pool % 2 != 1 or pool < 1:
        raise ValueError("the pooling window must be odd")
    h = pool // 2
    out = np.empty(n_cand, dtype=np.float32)
    for i in range(n_cand):
        out[i] = s[max(0, i - h):min(n_cand, i + h + 1)].max()
    return out


def normalised_scores(s: np.ndarray, n_cand: int) -> np.ndarray:
    """s~_i = s_i / max_j s_j over the candidates, the maximum clamped to >= 1e-12 (Eq. (5), R7, R8)."""
    den = max(float(s[:n_cand].max()), float(f32(NORMALISER_FLOOR)))
    return (s[:n_cand].astype(np.float32) / np.float32(den)).astype(np.float32)


def top_candidates(s: np.ndarray, n_cand: int, n_keep: int) -> List[int]:
    """Positions of the n_keep largest base scores among [0, n_cand), ties to the lower position
    (section 3.2, top-4B restriction; R10).  Returned in ascending position order."""
    ranked = sorted(range(n_cand), key=lambda i: (-float(s[i]), i))
    return sorted(ranked[:n_keep])


def unit_keys(k_rows: np.ndarray) -> np.ndarray:
    """k / ||k|| per row, 0 for a zero row (R12)."""
    norms = np.sqrt((k_rows * k_rows).sum(axis=1))
    out = np.zeros_like(k_rows)
    nz = norms > 0
    out[nz] = k_rows[nz] / norms[nz, None]
    return out


@dataclasses.dataclass
class GreedyTrace:
    selected: List[int]          # admission order
    score: List[float]           # winning s~ + lambda2 corr at each step (fp32 value)
    runner_up: List[Optional[int]]
    runner_up_score: List[float]
    corr: dict                   # final corr(i, S) over the candidates (fp32), by position
    best_corr: List[float] = dataclasses.field(default_factory=list)       # corr of the winner
    runner_up_corr: List[float] = dataclasses.field(default_factory=list)  # and of the runner-up


def greedy_mmr(s_tilde: np.ndarray, k_unit: np.ndarray, cand: List[int], lam2: float,
               budget: int) -> GreedyTrace:
    """Greedy admission (Eq. (5) second line, with Eq. (4)): B times, admit the candidate outside S
    with the largest s~_i + lambda2 corr(i, S); corr(i, S) = max(0, max_{j in S} cos(k_i, k_j)).

    The running maximum is updated only against the newly admitted key (R11); cosines are float64
    dot products of unit keys rounded to fp32; the score is a fp32 multiply-add; ties go to the lower
    position (R10).
    """
    lam = float(f32(lam2))
    corr = {i: np.float32(0.0) for i in cand}
    chosen: List[int] = []
    taken = set()
    trace = GreedyTrace([], [], [], [], {})
    for _ in range(budget):
        best = second = None
        best_v = second_v = -np.inf
        for i in cand:  # ascending positions: strict '>' keeps the lower position on ties
            if i in taken:
                continue
            v = float(f32(float(s_tilde[i]) + lam * float(corr[i])))
            if v > best_v:
                second, second_v = best, best_v
                best, best_v = i, v
            elif v > second_v:
                second, second_v = i, v
        if best is None:
            raise ValueError("budget exceeds the number of candidates")
        chosen.append(best)
        taken.add(best)
        trace.score.append(best_v)
        trace.runner_up.append(second)
        trace.runner_up_score.append(second_v)
        trace.best_corr.append(float(corr[best]))
        trace.runner_up_corr.append(float(corr[second]) if second is not None else 0.0)
        rest = [i for i in cand if i not in taken]
        if rest:
            cos = (k_unit[rest] @ k_unit[best]).astype(np.float32)
            for i, c in zip(rest, cos):
                if c > corr[i]:
                    corr[i] = c
    trace.selected = chosen
    trace.corr = {i: corr[i] for i in cand}
    return trace


# ------------------------------------------------------------------------------------------------
# Compaction (section 1 / 3.1: each layer keeps B entries; R5, R14)
# ------------------------------------------------------------------------------------------------

def kept_positions(selected: List[int], L: int, keep_tail: int) -> List[int]:
    return sorted(selected) + list(range(L - keep_tail, L))


def compact_rows(x: np.ndarray, keep: List[int]) -> np.ndarray:
    """Rows of one head's cache at the kept positions (x is [L, d], any dtype; exact copy)."""
    return np.stack([x[i] for i in keep])


# ------------------------------------------------------------------------------------------------
# One problem end to end
# ------------------------------------------------------------------------------------------------

@dataclasses.dataclass
class HeadResult:
    candidates: List[int]
    trace: GreedyTrace
    s: np.ndarray          # fp32 base scores over [0, n_cand)
    s_tilde: np.ndarray    # fp32 normalised scores over [0, n_cand)
    boundary_gap: Optional[tuple]  # (s of the last kept candidate, s of the first excluded)
    boundary_pos: Optional[tuple] = None  # their positions


@dataclasses.dataclass
class ProblemResult:
    row_max: np.ndarray    # [h_q, W]
    row_sum: np.ndarray    # [h_q, W]
    mu: np.ndarray         # [h_kv, L]
    sigma: np.ndarray      # [h_kv, L]
    heads: List[HeadResult]
    k_out: Optional[np.ndarray] = None  # [h_kv, B + keep_tail, d] as stored
    v_out: Optional[np.ndarray] = None
    attn: Optional[np.ndarray] = None   # [h_q, W, L]


def candidate_count(n_cand: int, budget: int, cand_mult: int) -> int:
    return n_cand if cand_mult == 0 else min(cand_mult * budget, n_cand)


def select_head(mu_g: np.ndarray, sigma_g: np.ndarray, k_g: np.ndarray, lam1: float, lam2: float,
                budget: int, n_cand: int, cand_mult: int = 4, pool: int = 1,
                w_mu: float = 1.0) -> HeadResult:
    """Selection for one kv head: base score (optionally max-pooled), normalisation, top-C
    restriction, greedy MMR."""
    s = base_scores(mu_g[:n_cand], sigma_g[:n_cand], lam1, w_mu)
    if pool > 1:
        s = max_pool(s, n_cand, pool)
    s_t = normalised_scores(s, n_cand)
    n_keep = candidate_count(n_cand, budget, cand_mult)
    cand = top_candidates(s, n_cand, n_keep)
    gap = pos = None
    if n_keep < n_cand:
        ranked = sorted(range(n_cand), key=lambda i: (-float(s[i]), i))
        gap = (float(s[ranked[n_keep - 1]]), float(s[ranked[n_keep]]))
        pos = (ranked[n_keep - 1], ranked[n_keep])
    k_unit = np.zeros_like(k_g)
    k_unit[cand] = unit_keys(k_g[cand])
    trace = greedy_mmr(s_t, k_unit, cand, lam2, budget)
    return HeadResult(cand, trace, s, s_t, gap, pos)


def evict_problem(q_win, k, v, dtype: str, scale: float, lam1: float, lam2: float, budget: int,
                  cand_mult: int = 4, keep_tail: Optional[int] = None, heads=None,
                  want_attn: bool = False, pool: int = 1, w_mu: float = 1.0,
                  sigma_all_rows: bool = False) -> ProblemResult:
    """Whole path for one problem (one layer of one sequence).

    q_win [h_q, W, d], k and v [h_kv, L, d] as stored (fp32 or bf16 bits).  `heads` restricts the
    selection to some kv heads (statistics are still returned for all of them).  pool / w_mu:
    see max_pool and base_scores; sigma_all_rows: the R1b reading of token_statistics.
    """
    qd = decode(q_win, dtype)
    kd = decode(k, dtype)
    h_q, w, _ = qd.shape
    h_kv, L, _ = kd.shape
    tail = w if keep_tail is None else keep_tail
    n_cand = L - tail
    group = h_q // h_kv
    row_max = np.empty((h_q, w))
    row_sum = np.empty((h_q, w))
    mu = np.empty((h_kv, L))
    sigma = np.empty((h_kv, L))
    attn = np.empty((h_q, w, L)) if want_attn else None
    for g in range(h_kv):  # one kv head at a time bounds the memory of the attention rows
        hs = slice(g * group, (g + 1) * group)
        lg = window_logits(qd[hs], kd[g:g + 1], scale)
        row_max[hs], row_sum[hs] = window_row_stats(lg)
        a = window_attention(lg)
        if want_attn:
            attn[hs] = a
        mu[g:g + 1], sigma[g:g + 1] = token_statistics(a, 1, sigma_all_rows)
    sel_heads = range(h_kv) if heads is None else heads
    results = []
    for g in range(h_kv):
        if g in sel_heads:
            results.append(select_head(mu[g], sigma[g], kd[g], lam1, lam2, budget, n_cand, cand_mult,
                                       pool, w_mu))
        else:
            results.append(None)
    res = ProblemResult(row_max, row_sum, mu, sigma, results, attn=attn)
    if v is not None and heads is None:
        ko = []
        vo = []
        for g in range(h_kv):
            keep = kept_positions(results[g].trace.selected, L, tail)
            ko.append(compact_rows(np.asarray(k)[g], keep))
            vo.append(compact_rows(np.asarray(v)[g], keep))
        res.k_out = np.stack(ko)
        res.v_out = np.stack(vo)
    return res
