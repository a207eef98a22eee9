"""Pins of the CPU oracle against what the paper and the mathematics fix (no GPU needed).

Each test checks the oracle against something other than itself: an independent library routine
(scaled dot-product attention, `statistics`, a stable sort), a closed form, an invariant, a special
case the paper states, or a from-scratch brute force on tiny inputs.
"""
import json
import math
import os
import statistics
from fractions import Fraction

import numpy as np
import pytest
import torch
from hypothesis import given, settings, strategies as st

from oracle import budgets, evict, profiles

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand(shape, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


# ------------------------------------------------------------------------------------------------
# Window attention (section 3.1)
# ------------------------------------------------------------------------------------------------

@pytest.mark.parametrize("h_q,h_kv,w,L,d", [(2, 1, 8, 40, 16), (4, 2, 5, 23, 8), (8, 8, 3, 9, 4)])
def test_window_attention_matches_torch_sdpa(h_q, h_kv, w, L, d):
    """A equals torch's scaled dot-product attention of the last W positions with a causal mask,
    read out through identity values (out = A @ I)."""
    q = _rand((h_q, w, d), 1)
    k = _rand((h_kv, L, d), 2)
    scale = 1.0 / math.sqrt(d)
    attn = evict.window_attention(evict.window_logits(q, k, scale))
    group = h_q // h_kv
    kt = torch.from_numpy(np.repeat(k, group, axis=0))
    qt = torch.from_numpy(q)
    pos_q = torch.arange(L - w, L)[:, None]
    mask = torch.arange(L)[None, :] <= pos_q  # True = may attend
    eye = torch.eye(L, dtype=torch.float64).expand(h_q, L, L)
    ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, eye, attn_mask=mask, scale=scale)
    np.testing.assert_allclose(attn, ref.numpy(), rtol=1e-12, atol=1e-15)


def test_row_stats_identical_keys_closed_form():
    """All keys equal: the row maximum is the common logit and Z counts the visible keys."""
    L, w, d = 64, 8, 16
    q = _rand((2, w, d), 3)
    key = _rand((d,), 4)
    k = np.tile(key, (1, L, 1))
    scale = 0.25
    m, z = evict.window_row_stats(evict.window_logits(q, k, scale))
    np.testing.assert_allclose(m, scale * (q @ key), rtol=1e-14)
    np.testing.assert_allclose(z, np.tile(np.arange(L - w + 1, L + 1, dtype=float), (2, 1)), rtol=1e-14)


def _closed_form_identical(L, w, i):
    """Exact mu_i, sigma_i^2 when all keys are equal: row r sees L - W + r + 1 keys uniformly."""
    vals = [Fraction(1, L - w + r + 1) if i <= L - w + r else Fraction(0) for r in range(w)]
    mu = sum(vals) / w
    var = sum((v - mu) ** 2 for v in vals) / (w - 1)
    return mu, var


@pytest.mark.parametrize("L,w", [(512, 8), (100, 4), (33, 32)])
def test_mu_sigma_identical_keys_closed_form(L, w):
    """Eq. (1) and Eq. (3) against exact rational arithmetic for identical keys, for prefix tokens
    and for tokens inside the window (which only some rows see)."""
    d = 8
    q = _rand((1, w, d), 5)
    k = np.tile(_rand((d,), 6), (1, L, 1))
    attn = evict.window_attention(evict.window_logits(q, k, 1.0 / math.sqrt(d)))
    mu, sigma = evict.token_statistics(attn, 1)
    for i in [0, 1, L // 2, L - w, L - w + 1, L - 1]:
        emu, evar = _closed_form_identical(L, w, i)
        assert mu[0, i] == pytest.approx(float(emu), rel=1e-13)
        assert sigma[0, i] == pytest.approx(math.sqrt(float(evar)), rel=1e-9, abs=1e-300)


def test_mu_sigma_identical_keys_L512_W8_values():
    """Paper's window size |W| = 8 at L = 512: mu = 1.96660826849e-3, sigma = 9.4735468349e-6
    for every prefix token (values of the exact closed form above, to 12 digits)."""
    with open(os.path.join(GOLDEN, "paper_constants.json")) as f:
        assert json.load(f)["window_size"]["W"] == 8
    L, w, d = 512, 8, 8
    q = _rand((1, w, d), 7)
    k = np.tile(_rand((d,), 8), (1, L, 1))
    mu, sigma = evict.token_statistics(evict.window_attention(evict.window_logits(q, k, 0.3)), 1)
    assert mu[0, 0] == pytest.approx(1.96660826849e-3, rel=1e-11)
    assert sigma[0, 0] == pytest.approx(9.4735468349e-6, rel=1e-9)


def test_mu_sums_to_one():
    """Every attention row sums to one, so the mean over rows (Eq. (1)) sums to one over tokens."""
    q = _rand((8, 6, 16), 9)
    k = _rand((2, 50, 16), 10, 3.0)
    mu, _ = evict.token_statistics(evict.window_attention(evict.window_logits(q, k, 0.25)), 2)
    np.testing.assert_allclose(mu.sum(axis=1), 1.0, rtol=1e-13)


def test_mu_sigma_against_statistics_module():
    """Eq. (1) is the mean and Eq. (3) the sample standard deviation (divisor W - 1) over the window
    rows; with grouped heads the rows are first averaged over the group (reading R1)."""
    rng = np.random.default_rng(11)
    attn = rng.random((6, 5, 7))  # 6 query heads, 5 rows, 7 tokens; 3 kv heads of 2
    mu, sigma = evict.token_statistics(attn, 3)
    for g in range(3):
        for i in range(7):
            rows = [statistics.mean([attn[2 * g, r, i], attn[2 * g + 1, r, i]]) for r in range(5)]
            assert mu[g, i] == pytest.approx(statistics.mean(rows), rel=1e-13)
            assert sigma[g, i] == pytest.approx(statistics.stdev(rows), rel=1e-11)


def test_gqa_identical_group_heads_reduce_to_single_head():
    """If every query head of a group carries the same queries, grouped statistics equal the
    single-head Eq. (1) / Eq. (3) of one of them."""
    q1 = _rand((1, 6, 8), 12)
    k = _rand((1, 30, 8), 13, 2.0)
    single = evict.token_statistics(evict.window_attention(evict.window_logits(q1, k, 0.35)), 1)
    q4 = np.repeat(q1, 4, axis=0)
    grouped = evict.token_statistics(evict.window_attention(evict.window_logits(q4, k, 0.35)), 1)
    np.testing.assert_allclose(grouped[0], single[0], rtol=1e-14)
    np.testing.assert_allclose(grouped[1], single[1], rtol=1e-12)


def test_all_rows_dispersion_against_statistics_module():
    """Reading R1b: the mean and the sample standard deviation over all G W (head, row) values."""
    rng = np.random.default_rng(31)
    attn = rng.random((6, 5, 7))  # 6 query heads, 5 rows, 7 tokens; 3 kv heads of 2
    mu, sigma = evict.token_statistics(attn, 3, all_rows=True)
    for g in range(3):
        for i in range(7):
            vals = [attn[h, r, i] for h in (2 * g, 2 * g + 1) for r in range(5)]
            assert mu[g, i] == pytest.approx(statistics.mean(vals), rel=1e-13)
            assert sigma[g, i] == pytest.approx(statistics.stdev(vals), rel=1e-11)


def test_all_rows_dispersion_single_head_and_identical_heads():
    """G = 1: both readings coincide.  G identical heads: the sum of squared deviations over the
    G W values is G times the one over W rows, so sigma_all^2 (G W - 1) = G (W - 1) sigma^2, and
    the means agree."""
    q1 = _rand((1, 6, 8), 32)
    k = _rand((1, 30, 8), 33, 2.0)
    a1 = evict.window_attention(evict.window_logits(q1, k, 0.35))
    np.testing.assert_array_equal(evict.token_statistics(a1, 1, all_rows=True)[1],
                                  evict.token_statistics(a1, 1)[1])
    G, w = 4, 6
    a4 = evict.window_attention(evict.window_logits(np.repeat(q1, G, axis=0), k, 0.35))
    mu_g, sg_g = evict.token_statistics(a4, 1)
    mu_a, sg_a = evict.token_statistics(a4, 1, all_rows=True)
    np.testing.assert_allclose(mu_a, mu_g, rtol=1e-14)
    np.testing.assert_allclose(sg_a ** 2 * (G * w - 1), G * (w - 1) * sg_g ** 2, rtol=1e-12)


def test_all_rows_dispersion_law_of_total_variance():
    """sum_{h,r} (A - mu)^2 = sum_{h,r} (A_hr - a_r)^2 + G sum_r (a_r - mu)^2 with a_r the group
    mean of row r: ties the two readings together on unequal heads."""
    q = _rand((4, 5, 8), 34)
    k = _rand((1, 25, 8), 35, 2.0)
    attn = evict.window_attention(evict.window_logits(q, k, 0.4))
    G, w = 4, 5
    _, sg_g = evict.token_statistics(attn, 1)
    _, sg_a = evict.token_statistics(attn, 1, all_rows=True)
    a_r = attn.mean(axis=0)
    within = ((attn - a_r[None]) ** 2).sum(axis=(0, 1))
    np.testing.assert_allclose(sg_a[0] ** 2 * (G * w - 1), within + G * (w - 1) * sg_g[0] ** 2,
                               rtol=1e-11)


def test_causal_mask_window_tokens():
    """Window row r sees keys up to L - W + r (reading R2): the last key gets attention only from
    the last row, so its mean is A[last row, L-1] / W."""
    q = _rand((1, 4, 8), 14)
    k = _rand((1, 20, 8), 15)
    attn = evict.window_attention(evict.window_logits(q, k, 0.3))
    for r in range(4):
        assert np.all(attn[0, r, 16 + r + 1:] == 0.0)
        assert np.all(attn[0, r, :16 + r + 1] > 0.0)
    mu, _ = evict.token_statistics(attn, 1)
    assert mu[0, 19] == pytest.approx(attn[0, 3, 19] / 4, rel=1e-14)


def test_decode_bf16_exact():
    bits = np.array([0x3F80, 0xC000, 0x0000, 0x3E20, 0x7F7F], dtype=np.uint16)
    np.testing.assert_array_equal(evict.decode(bits, "bf16"),
                                  [1.0, -2.0, 0.0, 0.15625, 3.3895313892515355e38])


# ------------------------------------------------------------------------------------------------
# Base score, normalisation, candidate restriction (section 3.2)
# ------------------------------------------------------------------------------------------------

def test_normalised_scores_bounds_and_ranking():
    """s~ = s / max s: the maximum becomes 1, s~ lies in [0, 1] when lambda1 >= 0, and the ranking
    is preserved (section 3.2 after Eq. (5))."""
    rng = np.random.default_rng(16)
    mu, sg = rng.random(100) * 1e-3, rng.random(100) * 1e-4
    s = evict.base_scores(mu, sg, 0.7)
    st_ = evict.normalised_scores(s, 100)
    assert st_.max() == np.float32(1.0)
    assert st_.min() >= 0.0
    assert list(np.argsort(-s, kind="stable")) == list(np.argsort(-st_, kind="stable"))


def test_normaliser_clamped_positive():
    """All base scores non-positive: the normaliser falls back to its positive floor (R7), so the
    order is preserved and nothing divides by zero (section 3.2, Eq. (5))."""
    s = np.array([-3e-4, -1e-4, 0.0, -2e-4], dtype=np.float32)
    st_ = evict.normalised_scores(s, 4)
    assert np.all(np.isfinite(st_))
    assert list(np.argsort(-st_, kind="stable")) == [2, 1, 3, 0]


def test_base_score_is_fp32_fma():
    """s = mu + lambda1 sigma, rounded once to fp32."""
    mu = np.array([1.0 / 3.0])
    sg = np.array([2.0 / 7.0])
    s = evict.base_scores(mu, sg, 0.1)
    exact = float(np.float32(1.0 / 3.0)) + float(np.float32(0.1)) * float(np.float32(2.0 / 7.0))
    assert s[0] == np.float32(exact)


@given(st.lists(st.integers(0, 6), min_size=1, max_size=30), st.integers(1, 30))
@settings(max_examples=60, deadline=None)
def test_top_candidates_matches_stable_topk(vals, n_keep):
    """Top-C by base score with ties to the lower position equals a stable descending sort, and a
    brute-force count: i is kept iff fewer than C positions beat it (higher score, or equal score at
    a lower position)."""
    s = np.asarray(vals, dtype=np.float32) * np.float32(0.25)
    n = len(vals)
    n_keep = min(n_keep, n)
    got = evict.top_candidates(s, n, n_keep)
    ref = sorted(np.argsort(-s, kind="stable")[:n_keep].tolist())
    assert got == ref
    brute = [i for i in range(n)
             if sum(1 for j in range(n) if s[j] > s[i] or (s[j] == s[i] and j < i)) < n_keep]
    assert got == brute


def test_candidate_count_is_four_budget():
    with open(os.path.join(GOLDEN, "paper_constants.json")) as f:
        mult = json.load(f)["candidate_multiple"]["cand_mult"]
    assert evict.candidate_count(10000, 64, mult) == 256
    assert evict.candidate_count(100, 64, mult) == 100
    assert evict.candidate_count(10000, 64, 0) == 10000


# ------------------------------------------------------------------------------------------------
# Greedy MMR admission (Eq. (2), (4), (5))
# ------------------------------------------------------------------------------------------------

def _brute_greedy(s_tilde, k_unit, cand, lam2, budget):
    """From scratch at every step: corr(i, S) = max(0, max_{j in S} cos(k_i, k_j)), corr(i, {}) = 0;
    argmax of s~ + lambda2 corr over i outside S, ties to the lower position.  Plain Python floats,
    with the same fp32 rounding of cosines and scores as the decision precision."""
    S = []
    lam = float(np.float32(lam2))
    for _ in range(budget):
        best, best_v = None, None
        for i in sorted(cand):
            if i in S:
                continue
            corr = 0.0
            for j in S:
                c = float(np.float32(sum(float(a) * float(b) for a, b in zip(k_unit[i], k_unit[j]))))
                corr = max(corr, c)
            v = float(np.float32(float(s_tilde[i]) + lam * corr))
            if best_v is None or v > best_v:
                best, best_v = i, v
        S.append(best)
    return S


@given(st.integers(0, 10_000), st.integers(2, 12), st.integers(1, 8),
       st.sampled_from([-1.5, -0.8, -0.15, 0.0, 0.4, 2.0]))
@settings(max_examples=40, deadline=None)
def test_greedy_matches_bruteforce(seed, n, budget, lam2):
    """The incremental running-max greedy equals a from-scratch recomputation of corr at every step
    (spec pin: exhaustive brute-force greedy on tiny inputs)."""
    budget = min(budget, n)
    rng = np.random.default_rng(seed)
    s_t = rng.random(n).astype(np.float32)
    k_unit = evict.unit_keys(rng.standard_normal((n, 5)))
    cand = list(range(n))
    tr = evict.greedy_mmr(s_t, k_unit, cand, lam2, budget)
    assert tr.selected == _brute_greedy(s_t, k_unit, cand, lam2, budget)


def test_greedy_zero_lambdas_is_top_b_by_mean():
    """lambda1 = lambda2 = 0 reduces the score to mean attention alone: the B tokens with the
    largest mu, admitted in descending order of mu (section 3.2, Eq. (5))."""
    rng = np.random.default_rng(17)
    mu = rng.random(300) * 1e-3
    sg = rng.random(300) * 1e-3
    k = rng.standard_normal((300, 16))
    h = evict.select_head(mu, sg, k, 0.0, 0.0, 20, 300)
    ref = np.argsort(-mu.astype(np.float32), kind="stable")[:20].tolist()
    assert h.trace.selected == ref


def test_greedy_lambda2_zero_is_top_b_by_base_score():
    rng = np.random.default_rng(18)
    mu = rng.random(200) * 1e-3
    sg = rng.random(200) * 1e-3
    k = rng.standard_normal((200, 16))
    h = evict.select_head(mu, sg, k, 0.6, 0.0, 15, 200)
    s = mu.astype(np.float32).astype(np.float64) + float(np.float32(0.6)) * sg.astype(np.float32)
    ref = np.argsort(-s.astype(np.float32), kind="stable")[:15].tolist()
    assert h.trace.selected == ref


def test_first_pick_maximises_normalised_score():
    """The first admission maximises s~ (section 3.2, after Eq. (5)) for any lambda2."""
    rng = np.random.default_rng(19)
    for lam2 in (-3.0, -0.15, 0.5, 3.0):
        mu = rng.random(120) * 1e-3
        sg = rng.random(120) * 1e-3
        k = rng.standard_normal((120, 8))
        h = evict.select_head(mu, sg, k, 0.3, lam2, 10, 120)
        assert h.trace.selected[0] == int(np.argmax(h.s_tilde))


def test_non_positive_cosines_are_clamped():
    """Keys that are pairwise orthogonal or opposite (+-e_i) have corr = 0 after the clamp of
    Eq. (4), so any lambda2 gives top-B by s."""
    d = 16
    basis = np.concatenate([np.eye(d), -np.eye(d)])  # 32 keys, cosines 0 or -1
    rng = np.random.default_rng(20)
    mu = rng.random(32) * 1e-3
    sg = np.zeros(32)
    for lam2 in (-2.0, 2.0):
        h = evict.select_head(mu, sg, basis, 0.0, lam2, 12, 32)
        assert h.trace.selected == np.argsort(-mu.astype(np.float32), kind="stable")[:12].tolist()
        assert all(v == 0.0 for v in h.trace.corr.values())


def test_positive_lambda2_walks_along_an_arc():
    """lambda2 > 0 rewards similarity (section 3.2 after Eq. (4)): with keys on a one-sided arc and
    nearly equal base scores, each admission after the first is the nearest remaining angle."""
    n = 10
    ang = np.linspace(0.0, 1.2, n)
    k = np.stack([np.cos(ang), np.sin(ang), np.zeros(n)], axis=1)
    # first pick: angle 0; the other base scores grow with the angle, so without the set term the
    # order would run backwards along the arc
    s_t = np.float32(0.9) + np.arange(n, dtype=np.float32) * np.float32(1e-3)
    s_t[0] = 1.0
    tr = evict.greedy_mmr(s_t, evict.unit_keys(k), list(range(n)), 5.0, n)
    assert tr.selected == list(range(n))
    assert evict.greedy_mmr(s_t, evict.unit_keys(k), list(range(n)), 0.0, n).selected == \
        [0] + list(range(n - 1, 0, -1))


def test_mmr_hand_worked_example():
    """Two near-duplicates A, A' and a different token C (Eq. (4)-(5), lambda2 = -0.5).
    s~: A = 1.0, A' = 0.99, C = 0.9; cos(A, A') = 0.98, cos(A, C) = cos(A', C) = 0.
      step 1: A (largest s~);
      step 2: A' scores 0.99 - 0.5 * 0.98 = 0.50, C scores 0.9 - 0 = 0.9   -> C;
      step 3: A' (only one left).
    With lambda2 = 0 the order is A, A', C instead."""
    c = 0.98
    k = np.array([[1.0, 0.0, 0.0], [c, math.sqrt(1 - c * c), 0.0], [0.0, 0.0, 1.0]])
    s_t = np.array([1.0, 0.99, 0.9], dtype=np.float32)
    assert evict.greedy_mmr(s_t, k, [0, 1, 2], -0.5, 3).selected == [0, 2, 1]
    assert evict.greedy_mmr(s_t, k, [0, 1, 2], 0.0, 3).selected == [0, 1, 2]
    tr = evict.greedy_mmr(s_t, k, [0, 1, 2], -0.5, 2)
    assert tr.score[1] == pytest.approx(0.9)
    assert float(tr.corr[1]) == pytest.approx(0.98, rel=1e-6)


def test_zero_key_has_zero_cosine():
    k = np.array([[0.0, 0.0], [1.0, 0.0], [1.0, 1e-9]])
    u = evict.unit_keys(k)
    assert np.all(u[0] == 0.0)
    tr = evict.greedy_mmr(np.array([0.5, 1.0, 0.9], dtype=np.float32), u, [0, 1, 2], -1.0, 3)
    assert tr.selected == [1, 0, 2]  # the zero key is not penalised; the duplicate of 1 is


def test_ties_go_to_lower_position():
    s_t = np.array([0.5, 0.7, 0.7, 0.7], dtype=np.float32)
    k = evict.unit_keys(np.eye(4))
    assert evict.greedy_mmr(s_t, k, [0, 1, 2, 3], -1.0, 4).selected == [1, 2, 3, 0]
    assert evict.top_candidates(np.array([1, 2, 2, 2], dtype=np.float32), 4, 2) == [1, 2]


# ------------------------------------------------------------------------------------------------
# Compaction
# ------------------------------------------------------------------------------------------------

# ------------------------------------------------------------------------------------------------
# Max-pooling of the base score and the mean-free score (NEXT items of the hot path)
# ------------------------------------------------------------------------------------------------

@pytest.mark.parametrize("pool", [1, 3, 5, 7, 31])
def test_max_pool_matches_scipy_filter(pool):
    """The pooled score equals scipy's 1-D maximum filter with the outside counted as -inf."""
    from scipy.ndimage import maximum_filter1d
    s = _rand(300, 21).astype(np.float32)
    ref = maximum_filter1d(s.astype(np.float64), size=pool, mode="constant", cval=-np.inf)
    np.testing.assert_array_equal(evict.max_pool(s, 300, pool), ref.astype(np.float32))


def test_max_pool_spreads_a_spike_and_stops_at_the_candidate_range():
    s = np.zeros(20, dtype=np.float32)
    s[10] = 5.0
    s[19] = 9.0                     # outside the candidate range [0, 18)
    out = evict.max_pool(s, 18, 5)
    assert list(np.flatnonzero(out == 5.0)) == [8, 9, 10, 11, 12]
    assert out.max() == 5.0 and len(out) == 18
    with pytest.raises(ValueError):
        evict.max_pool(s, 18, 4)


def test_pooled_selection_with_zero_lambdas_is_top_b_of_the_pooled_mean():
    """lambda1 = lambda2 = 0 with pooling: the admissions are the B largest pooled means (ties to
    the lower position), found here by a sort of the brute-force window maxima."""
    rng = np.random.default_rng(7)
    n, B, pool = 60, 9, 5
    mu = rng.random(n).astype(np.float32)
    k = rng.standard_normal((n, 8))
    res = evict.select_head(mu, np.zeros(n), k, 0.0, 0.0, B, n, cand_mult=0, pool=pool)
    pooled = [max(mu[max(0, i - 2):min(n, i + 3)]) for i in range(n)]
    want = sorted(range(n), key=lambda i: (-pooled[i], i))[:B]
    assert res.trace.selected == want


def test_mean_free_score_with_lambda1_one_is_sigma():
    """w_mu = 0, lambda1 = 1: the base score is sigma itself (rounded to fp32)."""
    rng = np.random.default_rng(8)
    mu, sg = rng.random(50), rng.random(50)
    np.testing.assert_array_equal(evict.base_scores(mu, sg, 1.0, w_mu=0.0), sg.astype(np.float32))
    np.testing.assert_array_equal(evict.base_scores(mu, sg, 0.4, w_mu=1.0),
                                  evict.base_scores(mu, sg, 0.4))


def test_mean_free_selection_with_lambda2_zero_is_top_b_by_sigma():
    rng = np.random.default_rng(9)
    n, B = 40, 6
    mu, sg = rng.random(n), rng.random(n)
    res = evict.select_head(mu, sg, rng.standard_normal((n, 4)), 0.7, 0.0, B, n, cand_mult=0,
                            w_mu=0.0)
    want = sorted(range(n), key=lambda i: (-float(np.float32(sg[i])), i))[:B]
    assert res.trace.selected == want


def test_compaction_keeps_sorted_selection_then_tail():
    L, d = 40, 4
    k = np.arange(L * d, dtype=np.uint16).reshape(L, d)
    keep = evict.kept_positions([30, 3, 17], L, 5)
    assert keep == [3, 17, 30, 35, 36, 37, 38, 39]
    out = evict.compact_rows(k, keep)
    assert out.dtype == k.dtype
    np.testing.assert_array_equal(out[:, 0] // d, keep)


def test_evict_problem_end_to_end_tiny():
    """One small problem through every step; the compacted rows are the kept positions of the
    stored arrays, byte for byte."""
    rng = np.random.default_rng(21)
    q = rng.standard_normal((4, 6, 8)).astype(np.float32)
    k = rng.standard_normal((2, 50, 8)).astype(np.float32)
    v = rng.standard_normal((2, 50, 8)).astype(np.float32)
    res = evict.evict_problem(q, k, v, "f32", 0.35, 0.3, -0.5, 5)
    for g in range(2):
        sel = res.heads[g].trace.selected
        assert len(set(sel)) == 5 and all(0 <= i < 44 for i in sel)
        keep = sorted(sel) + list(range(44, 50))
        np.testing.assert_array_equal(res.k_out[g], k[g, keep])
        np.testing.assert_array_equal(res.v_out[g], v[g, keep])


# ------------------------------------------------------------------------------------------------
# Depth profiles (section 3.3, Eq. (6))
# ------------------------------------------------------------------------------------------------

def test_sinh_span_matches_paper():
    with open(os.path.join(GOLDEN, "paper_constants.json")) as f:
        g = json.load(f)["sinh_span"]
    lam = profiles.layer_lambdas("global", [g["a"]], 1)[0]
    assert lam == pytest.approx(g["lambda_approx"], abs=0.05)
    assert lam == pytest.approx((math.e ** 2 - math.e ** -2) / 2, rel=1e-15)
    assert profiles.layer_lambdas("global", [-g["a"]], 1)[0] == -lam
    assert profiles.layer_lambdas("global", [1e-4], 1)[0] == pytest.approx(1e-4, rel=1e-8)


def test_segments_thirds_of_32_layers():
    with open(os.path.join(GOLDEN, "paper_constants.json")) as f:
        seg = json.load(f)["segments"]
    n = seg["n_layers"]
    a = [0.1, 0.2, 0.3]
    lat = [profiles.latent("segments", a, layer, n) for layer in range(n)]
    assert lat[:11] == [0.1] * 11 and lat[11:22] == [0.2] * 11 and lat[22:] == [0.3] * 10


def test_global_is_a_special_case_of_segments_and_curve():
    n = 32
    glob = profiles.layer_lambdas("global", [-0.15], n)
    assert profiles.layer_lambdas("segments", [-0.15] * 3, n) == glob
    assert profiles.layer_lambdas("curve", [-0.15, 0.0, 0.0], n) == glob


def test_curve_endpoints_and_sign_flip():
    c0, c1, c2 = -1.47190, 6.19355, -6.0
    lam = profiles.layer_lambdas("curve", [c0, c1, c2], 32)
    assert lam[0] == pytest.approx(math.sinh(c0))
    assert lam[31] == pytest.approx(math.sinh(c0 + c1 + c2))
    positive = [layer for layer in range(32) if lam[layer] > 0]
    assert positive == list(range(12, 21))


def test_profile_rejects_bad_arguments():
    with pytest.raises(ValueError):
        profiles.latent("curve", [1.0, 2.0], 0, 32)
    with pytest.raises(ValueError):
        profiles.latent("nope", [1.0], 0, 32)
    with pytest.raises(ValueError):
        profiles.latent("global", [1.0], 32, 32)


# ------------------------------------------------------------------------------------------------
# Depth-decreasing budgets at a fixed total (reading R26)
# ------------------------------------------------------------------------------------------------

def test_pyramid_budgets_hand_worked():
    """B = 10, beta = 5, 4 layers: B_min = 2, B_max = 18, real budgets 18, 12.67, 7.33, 2, rounded
    away from 10: 18, 13, 7, 2."""
    assert budgets.pyramid_budgets(10, 4, 5.0) == [18, 13, 7, 2]


def test_pyramid_budgets_benchmark_shape():
    """B = 64 over 32 layers with beta = 20: from 125 down to 3, total 2048, and the largest
    top-4B candidate set 4 * 125 = 500."""
    b = budgets.pyramid_budgets(64, 32, 20.0)
    assert b[0] == 125 and b[-1] == 3 and sum(b) == 2048


@settings(max_examples=300, deadline=None)
@given(st.integers(1, 300), st.integers(1, 48), st.sampled_from([1.0, 1.5, 2.0, 5.0, 20.0, 1e9]))
def test_pyramid_budgets_invariants(B, n, beta):
    """Same total as the uniform allocation, non-increasing with depth, mirror-symmetric about B,
    within [B_min, B_max], and uniform for beta = 1 or a single layer."""
    b = budgets.pyramid_budgets(B, n, beta)
    assert len(b) == n and sum(b) == n * B
    assert all(x >= y for x, y in zip(b, b[1:]))
    assert all(b[i] + b[n - 1 - i] == 2 * B for i in range(n))
    b_min = max(1, math.floor(B / beta))
    assert all(b_min <= x <= 2 * B - b_min for x in b)
    if beta == 1.0 or n == 1:
        assert b == [B] * n
    if n > 1:
        assert b[0] == 2 * B - b_min and b[-1] == b_min


# ------------------------------------------------------------------------------------------------
# Decode attention over the compacted cache
# ------------------------------------------------------------------------------------------------

def test_decode_attention_against_sdpa():
    """GQA decode (8 query heads on 2 kv heads, one query token) against torch's scaled dot-product
    attention in float64 with the kv heads repeated per group."""
    from oracle import decode
    rng = np.random.default_rng(41)
    q = rng.standard_normal((8, 16))
    k = rng.standard_normal((2, 37, 16))
    v = rng.standard_normal((2, 37, 16))
    o = decode.decode_attention(q, k, v, 0.3)
    kt = torch.from_numpy(np.repeat(k, 4, axis=0))
    vt = torch.from_numpy(np.repeat(v, 4, axis=0))
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[:, None, :], kt, vt, scale=0.3)[:, 0, :].numpy()
    np.testing.assert_allclose(o, ref, rtol=1e-12, atol=1e-12)


def test_decode_attention_special_cases():
    """Identical keys average the values; one row returns its value; a key far along the query
    returns (nearly) its value; appending k_new / v_new equals attending over the longer cache."""
    from oracle import decode
    rng = np.random.default_rng(42)
    q = rng.standard_normal((2, 8))
    v = rng.standard_normal((1, 10, 8))
    k_same = np.tile(rng.standard_normal(8), (1, 10, 1))
    np.testing.assert_allclose(decode.decode_attention(q, k_same, v, 0.5),
                               np.tile(v[0].mean(axis=0), (2, 1)), rtol=1e-13)
    np.testing.assert_allclose(decode.decode_attention(q, k_same[:, :1], v[:, :1], 0.5),
                               np.tile(v[0, 0], (2, 1)), rtol=1e-15)
    k = rng.standard_normal((1, 10, 8)) * 0.01
    k[0, 6] = 400.0 * q[0] / np.linalg.norm(q[0])
    o = decode.decode_attention(q[:1], k, v, 1.0)
    np.testing.assert_allclose(o[0], v[0, 6], rtol=1e-9, atol=1e-9)
    k2 = rng.standard_normal((1, 10, 8))
    a = decode.decode_attention(q, k2[:, :9], v[:, :9], 0.4, k2[:, 9], v[:, 9])
    np.testing.assert_array_equal(a, decode.decode_attention(q, k2, v, 0.4))
