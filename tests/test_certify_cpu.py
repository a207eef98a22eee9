"""CPU checks of the margin certification (tests/certify.py) and of the stored certified inputs."""
import numpy as np

from oracle import evict
from paper_2609_30738_amd import workloads
from tests import certified_cases, certify


def _head(s, k, lam2=-0.5, budget=2, n_keep=3):
    n = len(s)
    s = np.asarray(s, dtype=np.float32)
    return evict.select_head(s.astype(np.float64), np.zeros(n), k, 0.0, lam2, budget, n,
                             cand_mult=n_keep // budget if n_keep % budget == 0 else 0)


def test_redraw_replaces_only_the_given_rows():
    wl = workloads.mistral_layer()
    wl.seq_lens = [1000]
    a = workloads.draw_problem(wl, 0)
    b = workloads.draw_problem(wl, 0, redraw={3: [100, 100, 700], 5: [9]})
    diff = np.argwhere((a.k != b.k).any(axis=2))
    assert diff.tolist() == [[3, 100], [3, 700], [5, 9]]
    c = workloads.draw_problem(wl, 0, redraw={3: [100]})
    assert not np.array_equal(b.k[3, 100], c.k[3, 100])  # the second re-draw of 100 differs
    assert np.array_equal(a.q_win, b.q_win) and np.array_equal(a.v, b.v)


def test_boundary_margin_detected_and_repaired():
    """Two tokens 1e-6 apart (relative) straddle the top-4 cut: the lower-ranked one is re-drawn."""
    rng = np.random.default_rng(0)
    k = rng.standard_normal((8, 16)).astype(np.float32)
    s = [1.0, 0.9, 0.8, 0.5, 0.5 * (1 - 1e-6), 0.1, 0.05, 0.01]
    h = _head(s, k, n_keep=4)
    c = certify.certify_head(h, k, -0.5, workloads.F32)
    assert c.boundary == "repair" and c.redraw[:1] == [4]
    s[4] = 0.3
    c = certify.certify_head(_head(s, k, n_keep=4), k, -0.5, workloads.F32)
    assert c.boundary == "certified"


def test_greedy_margin_detected_and_identical_keys_exempt():
    """Orthogonal keys, lambda2 < 0: the greedy ranks by s~; a near-tie between two different keys
    fails (the runner-up is re-drawn), an exact tie between identical keys does not."""
    k = np.eye(6, dtype=np.float32)
    s = [1.0, 0.7, 0.7 * (1 + 1e-7), 0.2, 0.1, 0.05]
    h = _head(s, k, budget=3, n_keep=6)
    c = certify.certify_head(h, k, -0.5, workloads.F32)
    assert c.greedy == "repair" and c.redraw == [1]
    k2 = k.copy()
    k2[2] = k2[1]
    s2 = [1.0, 0.7, 0.7, 0.25, 0.1, 0.05]
    h2 = _head(s2, k2, budget=3, n_keep=6)
    assert h2.trace.selected[:2] == [0, 1]  # the lower position wins the exact tie
    c2 = certify.certify_head(h2, k2, -0.5, workloads.F32)
    assert c2.ok and c2.exact_ties >= 1


def test_dense_cut_is_not_repaired():
    """A cut through many tokens with nearly equal scores (the flat bulk) is reported, not
    repaired."""
    rng = np.random.default_rng(1)
    k = rng.standard_normal((60, 16)).astype(np.float32)
    s = [1.0, 0.9] + [0.3 * (1 + 1e-7 * i) for i in range(58)]
    h = _head(s, k, budget=2, n_keep=8)
    c = certify.certify_head(h, k, -0.5, workloads.F32)
    assert c.boundary == "dense" and c.redraw == []


def test_stored_inputs_of_the_small_cases_are_certified():
    """The stored re-draws certify every head of the tiny fp32 layer, the Mistral-shaped layer and
    the exact-duplicates case (the oracle run again on the inputs drawn with them)."""
    for name in ("tiny_f32", "mistral_layer", "exact_duplicates"):
        wl = certified_cases.workload(name)
        red = certified_cases.load_redraw(name)
        opts = certified_cases.options(name)
        lam1, lam2 = certify.layer_lambdas(wl, range(wl.n_prob))
        for p in range(wl.n_prob):
            _, _, certs = certify.certify_problem(wl, p, p, float(lam1[p]), float(lam2[p]), opts,
                                                  red.get(p), repair=False)
            assert all(c.ok for c in certs), (name, p, certs)
