"""Margin certification of seeded inputs (test infrastructure: it runs only the CPU oracle).

The selection (section 3.2, Eq. (5) and the top-4B candidate restriction after it) is an integer
result decided by fp32 arithmetic.  The GPU path and the oracle compute the same statistics with
different rounding (fp32 against fp64), so they take the same decisions wherever every decision
has a margin larger than the error of the quantities it compares.  For one problem the oracle's
values must satisfy, per kv head:

  * candidate boundary:  s_(C) - s_(C+1) >= F eps_s (|s_(C)| + |s_(C+1)|)
  * every greedy step:   best - second >= F (eps_s (|s~_1| + |s~_2|) + eps_c |lambda2| (mc_1 + mc_2))

with eps_s = 1e-5 (relative error of a base score), eps_c = 1e-6 (absolute error of a cosine) and
F = 10; s are the base scores, s~ the normalised ones, mc the running maximum cosines of the two
competitors.  A pair of tokens with bitwise identical keys has identical statistics on both sides
and is decided by the lower position (R10) on both; it needs no margin.

With lambda2 = 0 the score is s~ alone and the admitted set is the top B by s~: only the last step
(the B-th admission against the best token left out) decides the set.

A head that fails is repaired by re-drawing the key of the lower-ranked token of the failing pair
(a fresh bulk key from a seed derived from its position, see workloads.draw_problem): at the
boundary every excluded token within the margin of s_(C), in the greedy the runner-up of the first
failing step.  The problem is then certified again, for at most 50 rounds.  Two cases are left
uncertified instead of repaired, because repairs cannot create the margin there: a boundary with
more than BAND_MAX tokens inside its margin (the cut falls inside the flat bulk of the scores,
where consecutive base scores differ by ~1e-7 relative), and a head whose repairs exceed
HEAD_REDRAW_CAP keys.  Such heads are compared by near-tie validity (tests/compare.py).  The
positions to re-draw depend only on the oracle's values; tests/golden/make_certified.py stores
them for the named workloads, and the tests check the margins again on the inputs they draw.
"""
from __future__ import annotations

import concurrent.futures
import dataclasses
import os
from typing import Callable, Dict, List, Optional, Sequence, Tuple

import numpy as np

from oracle import evict, profiles
from paper_2609_30738_amd import workloads

EPS_S = 1e-5
EPS_C = 1e-6
FACTOR = 10.0
MAX_ROUNDS = 50
BAND_MAX = 8          # more tokens than this within the boundary margin: the cut is in the bulk
HEAD_REDRAW_CAP = 64  # re-drawn keys per head before its certification is given up

Redraw = Dict[int, Dict[int, List[int]]]  # problem -> kv head -> positions (in re-draw order)


@dataclasses.dataclass
class Options:
    """Selection options of a certified case (those of the entry points' defaults unless set)."""
    cand_mult: int = 4
    keep_tail: Optional[int] = None
    pool: int = 1
    w_mu: float = 1.0
    sigma_all_rows: bool = False
    budgets: Optional[Tuple[int, ...]] = None  # per problem (index into the run's problems)

    def key(self) -> str:
        parts = []
        for f in dataclasses.fields(self):
            v = getattr(self, f.name)
            if v != f.default:
                parts.append(f"{f.name}={v}")
        return ",".join(parts)


@dataclasses.dataclass
class HeadCert:
    ok: bool                         # every decision certified (after this round's repairs)
    redraw: List[int]                # positions to re-draw this round
    boundary: str                    # "none" (no cut), "certified", "repair", "dense"
    greedy: str                      # "certified", "repair", "uncertified"
    boundary_ratio: Optional[float]  # margin / required margin at the candidate boundary
    step_ratio: Optional[float]      # smallest margin / required margin over the greedy steps
    exact_ties: int                  # decisions between identical keys (decided by position)


def layer_lambdas(wl: workloads.Workload, problems: Sequence[int]):
    """Per-problem fp32 coefficients from the oracle's profile evaluation (section 3.3)."""
    l1 = profiles.layer_lambdas(wl.lam1.family, wl.lam1.params, wl.n_layers)
    l2 = profiles.layer_lambdas(wl.lam2.family, wl.lam2.params, wl.n_layers)
    return (np.array([l1[wl.layer_of(p)] for p in problems], dtype=np.float32),
            np.array([l2[wl.layer_of(p)] for p in problems], dtype=np.float32))


def _same_key(k_head: np.ndarray, a: int, b: int) -> bool:
    return bool(np.array_equal(k_head[a], k_head[b]))


def _step_scores(h: evict.HeadResult, k_head: np.ndarray, lam2: float, t: int, dtype: str,
                 trace: evict.GreedyTrace, cand: Sequence[int]) -> Dict[int, float]:
    """fp32 scores s~ + lambda2 corr of the candidates still outside S before greedy step t,
    replayed from the trace's admissions with the oracle's formulas (used at exact ties only)."""
    cand = list(cand)
    kd = evict.decode(k_head[cand], dtype)
    ku = evict.unit_keys(kd)
    pos = {c: j for j, c in enumerate(cand)}
    corr = np.zeros(len(cand), dtype=np.float32)
    taken = np.zeros(len(cand), dtype=bool)
    for j in trace.selected[:t]:
        taken[pos[j]] = True
        cos = (ku @ ku[pos[j]]).astype(np.float32)
        upd = ~taken & (cos > corr)
        corr[upd] = cos[upd]
    lam = float(np.float32(lam2))
    return {c: float(np.float32(float(h.s_tilde[c]) + lam * float(corr[j])))
            for j, c in enumerate(cand) if not taken[j]}


def certify_boundary(h: evict.HeadResult, k_head: np.ndarray):
    """(status, ratio, positions to re-draw, exact ties) of the top-C candidate boundary."""
    if h.boundary_gap is None:
        return "none", None, [], 0
    v, s_next = h.boundary_gap
    pa, _ = h.boundary_pos
    need = FACTOR * EPS_S * (abs(v) + abs(s_next))
    s = np.asarray(h.s, dtype=np.float64)
    cand = set(h.candidates)
    # tokens with the boundary token's key (identical statistics, ordered by position on both
    # sides), and every other token, which must keep the margin from the boundary value
    band = [int(i) for i in np.flatnonzero(np.abs(s - v) < need)]
    tie = [i for i in band if _same_key(k_head, i, pa)]
    other = [i for i in band if i not in tie]
    straddle = any(i not in cand for i in tie)
    below = [i for i in other if i not in cand]
    above = [i for i in other if i in cand] if straddle else []
    gaps = [abs(float(s[i]) - v) for i in below + above]
    gap = min(gaps, default=need) if straddle else min([v - s_next] + gaps)
    ratio = gap / need if need > 0 else float("inf")
    ties = len(tie) - 1
    bad = below + ([pa] if above else [])
    if not bad:
        return "certified", ratio, [], ties
    if len(below) + len(above) > BAND_MAX:
        return "dense", ratio, [], ties  # the cut falls inside the flat bulk of the scores
    return "repair", ratio, sorted(set(bad)), ties


def certify_greedy(h: evict.HeadResult, k_head: np.ndarray, lam2: float, dtype: str,
                   trace: Optional[evict.GreedyTrace] = None, cand: Optional[Sequence[int]] = None):
    """(status, smallest ratio, position to re-draw or None, exact ties) of the greedy steps of
    `trace` over candidates `cand` (default: the oracle's own).  With lambda2 = 0 the score is s~
    alone and the admitted set is the top B by s~, so only the last step (the B-th against the
    (B+1)-th) decides the set; the order of the earlier steps is checked for validity instead."""
    tr = trace if trace is not None else h.trace
    cand = list(h.candidates if cand is None else cand)
    st = np.asarray(h.s_tilde, dtype=np.float64)
    lam = abs(float(np.float32(lam2)))
    steps = list(enumerate(zip(tr.selected, tr.runner_up)))
    if lam == 0.0:
        steps = steps[-1:]
    ratio_min = None
    ties = 0
    for t, (a, b) in steps:
        if b is None:
            continue
        need = FACTOR * (EPS_S * (abs(st[a]) + abs(st[b]))
                         + EPS_C * lam * (tr.best_corr[t] + tr.runner_up_corr[t]))
        gap = tr.score[t] - tr.runner_up_score[t]
        if gap == 0.0 and _same_key(k_head, a, b):
            # an exact tie between identical keys: the best competitor with another key must keep
            # the margin
            ties += 1
            sc = _step_scores(h, k_head, lam2, t, dtype, tr, cand)
            rest = [(v_, c) for c, v_ in sc.items() if not _same_key(k_head, c, a)]
            if not rest:
                continue
            v2, b = max(rest, key=lambda x: (x[0], -x[1]))
            gap = tr.score[t] - v2
            need = FACTOR * (EPS_S * (abs(st[a]) + abs(st[b])) + EPS_C * lam * 2.0)
        ratio = gap / need if need > 0 else float("inf")
        ratio_min = ratio if ratio_min is None else min(ratio_min, ratio)
        if gap < need:
            if lam == 0.0:
                # the B-th admission against every token left out: a cut through the bulk?
                taken = set(tr.selected)
                band = [c for c in cand if c not in taken and st[a] - st[c] < need]
                if len(band) > BAND_MAX:
                    return "dense", ratio_min, None, ties
            return "repair", ratio_min, int(b), ties  # later steps follow from a changed trace
    return "certified", ratio_min, None, ties


def certify_head(h: evict.HeadResult, k_head: np.ndarray, lam2: float,
                 dtype: str = workloads.BF16, redrawn: int = 0) -> HeadCert:
    """Check one head's decisions (the oracle's HeadResult) against the margins above.

    k_head: the head's stored keys [L, d] (bf16 bits or fp32), to recognise identical keys;
    redrawn: keys of this head re-drawn in earlier rounds (repairs stop at HEAD_REDRAW_CAP)."""
    b_stat, b_ratio, b_red, ties = certify_boundary(h, k_head)
    g_stat, g_ratio, g_red, g_ties = certify_greedy(h, k_head, lam2, dtype)
    redraw = list(b_red) + ([g_red] if g_red is not None else [])
    if redraw and redrawn + len(redraw) > HEAD_REDRAW_CAP:
        # give up on this head: it stays uncertified and is compared by near-tie validity
        redraw = []
        if b_stat == "repair":
            b_stat = "dense"
        if g_stat == "repair":
            g_stat = "uncertified"
    if g_stat == "dense":
        g_stat = "uncertified"
    ok = b_stat in ("none", "certified") and g_stat == "certified"
    return HeadCert(ok, redraw, b_stat, g_stat, b_ratio, g_ratio, ties + g_ties)


def run_oracle(wl: workloads.Workload, p: int, j: int, lam1: float, lam2: float,
               opts: Options, redraw_p: Optional[Dict[int, List[int]]] = None,
               inputs: Optional[workloads.ProblemInputs] = None, with_values: bool = False):
    """The oracle on problem p (j: its index among the run's problems, for per-problem budgets)."""
    pi = inputs if inputs is not None else workloads.draw_problem(wl, p, redraw=redraw_p)
    budget = wl.budget if opts.budgets is None else int(opts.budgets[j])
    res = evict.evict_problem(pi.q_win, pi.k, pi.v if with_values else None, wl.dtype, wl.scale,
                              float(lam1), float(lam2), budget, opts.cand_mult, opts.keep_tail,
                              pool=opts.pool, w_mu=opts.w_mu, sigma_all_rows=opts.sigma_all_rows)
    return pi, res


def certify_problem(wl: workloads.Workload, p: int, j: int, lam1: float, lam2: float,
                    opts: Options, redraw_p: Optional[Dict[int, List[int]]] = None,
                    repair: bool = True):
    """(p, {g: new positions to re-draw}, [HeadCert per head]); repair=False only assesses."""
    pi, res = run_oracle(wl, p, j, lam1, lam2, opts, redraw_p)
    L = pi.k.shape[1]
    k = pi.k
    if wl.dtype == workloads.BF16:
        k = k.view(np.uint16)
    certs = [certify_head(res.heads[g], k[g], lam2, wl.dtype,
                          len((redraw_p or {}).get(g, [])) if repair else HEAD_REDRAW_CAP + 1)
             for g in range(wl.h_kv)]
    new = {g: c.redraw for g, c in enumerate(certs) if c.redraw}
    for g, pos in new.items():
        assert all(0 <= x < L for x in pos)
    return p, new, certs


def _worker_init():
    try:
        from threadpoolctl import threadpool_limits
        threadpool_limits(1)
    except Exception:  # pragma: no cover
        pass


def _task(args):
    return certify_problem(*args)


def _pool(workers: int):
    return concurrent.futures.ProcessPoolExecutor(workers, initializer=_worker_init)


def default_workers() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def certify_workload(wl: workloads.Workload, problems: Optional[Sequence[int]] = None,
                     opts: Optional[Options] = None, redraw: Optional[Redraw] = None,
                     workers: Optional[int] = None, max_rounds: int = MAX_ROUNDS,
                     log: Callable[[str], None] = print):
    """Certify (and repair) the given problems; returns (redraw, rounds, certs by problem)."""
    opts = opts or Options()
    probs = list(range(wl.n_prob)) if problems is None else list(problems)
    lam1, lam2 = layer_lambdas(wl, probs)
    index = {p: j for j, p in enumerate(probs)}
    red: Redraw = {int(p): {int(g): list(v) for g, v in d.items()}
                   for p, d in (redraw or {}).items()}
    todo = list(probs)
    certs: Dict[int, List[HeadCert]] = {}
    workers = workers or default_workers()
    rounds = 0
    with _pool(workers) as ex:
        while todo:
            final = rounds >= max_rounds  # no more repairs: the last inputs are only assessed
            rounds += 1
            args = [(wl, p, index[p], float(lam1[index[p]]), float(lam2[index[p]]), opts,
                     red.get(p), not final) for p in todo]
            todo = []
            for p, new, cs in ex.map(_task, args):
                certs[p] = cs
                if new:
                    todo.append(p)
                    for g, pos in new.items():
                        red.setdefault(p, {}).setdefault(g, []).extend(pos)
            n_red = sum(len(v) for d in red.values() for v in d.values())
            log(f"  {wl.name}: round {rounds}: {len(todo)} problems to repair, "
                f"{n_red} keys re-drawn so far")
    return red, rounds, certs


def summarize(certs: Dict[int, List[HeadCert]]) -> str:
    flat = [c for cs in certs.values() for c in cs]
    br = [c.boundary_ratio for c in flat if c.boundary_ratio is not None and c.boundary != "dense"]
    sr = [c.step_ratio for c in flat if c.step_ratio is not None and c.greedy == "certified"]
    return (f"heads={len(flat)} certified={sum(c.ok for c in flat)} "
            f"boundary-in-bulk={sum(c.boundary == 'dense' for c in flat)} "
            f"greedy-certified={sum(c.greedy == 'certified' for c in flat)} "
            f"min-boundary-margin/required={min(br) if br else float('nan'):.3g} "
            f"min-step-margin/required={min(sr) if sr else float('nan'):.3g} "
            f"exact-ties={sum(c.exact_ties for c in flat)}")
