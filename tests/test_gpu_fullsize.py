"""GPU parity at the full workload sizes, in the benchmark's launch configuration (every layer of
every sequence in one batch; kv_window_candidates, then kv_mmr_select_candidates with the
compaction, and on the same inputs the other scoring routes and kv_mmr_select_ex for the optional
outputs), against the oracle on every problem and kv head (the ragged batch: every problem of two
whole sequences).  Inputs carry their stored margin
certification (tests/certify.py): a head whose cut and greedy the oracle certifies must reproduce
the oracle exactly; the summary line reports how many are.

Every output of the batch is also checked for properties that hold at any size: admitted positions
are distinct candidates, the candidate lists are ascending, sum_i mu_i = 1 per head, and the
compacted tail equals the last W rows.
"""
import numpy as np
import pytest

from paper_2609_30738_amd import workloads
from tests import gpu_cases
from tests.certified_cases import RAGGED_COMPARED_SEQS

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def _properties(run):
    wl = run.wl
    H = run.host
    B = run.budget
    n = len(run.problems)
    stride = H["cand_idx"].size // (n * wl.h_kv)
    sel = H["sel_idx"].reshape(n, wl.h_kv, B)
    cand = H["cand_idx"].reshape(n, wl.h_kv, stride)
    for j in range(n):
        L = int(run.packed.lens[j])
        tok = int(run.packed.tok_off[j])
        mu = H["mu"][tok * wl.h_kv:(tok + L) * wl.h_kv].reshape(wl.h_kv, L)
        np.testing.assert_allclose(mu.astype(np.float64).sum(axis=1), 1.0, rtol=2e-4,
                                   err_msg=f"problem {j}: sum of mu")
        for g in range(wl.h_kv):
            s = sel[j, g]
            c = cand[j, g]
            live = c[c >= 0]
            assert len(set(s.tolist())) == B
            assert np.all(np.diff(live) > 0)
            assert set(s.tolist()) <= set(live.tolist())
            assert np.all((s >= 0) & (s < L - wl.w))
    rows = B + wl.w
    ko = H["k_out"].reshape(n, wl.h_kv, rows, wl.d)
    for j in range(n):
        q, k, v = gpu_cases.problem_arrays(run, j)
        L = int(run.packed.lens[j])
        np.testing.assert_array_equal(ko[j, :, B:], k[:, L - wl.w:])


def _compare(run, js=None, all_certified=False):
    reports = gpu_cases.check_all(run, js)
    print("  ", gpu_cases.summarize(reports), flush=True)
    if all_certified:
        assert all(r.certified for r in reports), gpu_cases.summarize(reports)
    return reports


def test_headline_32_layers_L32768():
    """32 layers x L=32768, W=32, B=64, quadratic lambda2 profile (the benchmark workload): all 256
    (layer, kv head) units against the oracle, through the benchmark's calls."""
    run = gpu_cases.run_case("pass_32k", timed=True)
    _properties(run)
    _compare(run, all_certified=True)


@pytest.mark.parametrize("budget", [32, 64, 128])
def test_32_layers_L8192_segments(budget):
    """32 layers x L=8192, three-segment lambda2, B in {32, 64, 128}: every unit, benchmark calls."""
    run = gpu_cases.run_case(f"pass_8k_B{budget}", timed=True)
    _properties(run)
    _compare(run)


@pytest.mark.parametrize("lam_run", ["dispersion_only", "redundancy_only", "both"])
def test_ragged_8x32(lam_run):
    """8 sequences (L ~ U{2048..31744}) x 32 layers, B=128, the three term-ablation runs (section
    4.3, Table 3): the whole batch on the GPU, every unit of sequences 1 (30053 keys) and 7 (4448
    keys) against the oracle."""
    run = gpu_cases.run_case(f"ragged_{lam_run}", timed=True)
    _properties(run)
    wl = run.wl
    js = [j for j, p in enumerate(run.problems) if wl.seq_of(p) in RAGGED_COMPARED_SEQS]
    _compare(run, js)


@pytest.mark.parametrize("pool", [1, 5])
def test_long_context_select_from_global_scores(pool):
    """L = 40000 > the 34816 candidate scores the selection stages in LDS: the score keys are
    re-formed from mu / sigma in HBM on every pass (and pooled there), 2 layers."""
    wl = workloads.mistral_layer()
    wl.seq_lens = [40000]
    wl.n_layers = 2
    run = gpu_cases.run_gpu(wl, fused=True, pool=pool)
    _properties(run)
    _compare(run)


def test_32_layers_L8192_unfused_one_segment_per_unit():
    """kv_window_scores, then kv_mu_sigma from its row statistics, on the whole 32-layer batch:
    every unit is one segment, so the first pass writes the row statistics itself."""
    run = gpu_cases.run_case("pass_8k_B64", fused=False)
    _properties(run)
    _compare(run, [0, 15, 31])


@pytest.mark.parametrize("fused", [True, False])
def test_one_layer_of_the_32k_pass_alone(fused):
    """One layer of the L=32768 workload launched by itself, as in the per-layer schedule: 32
    segments of 1024 keys per unit, whose partials the second pass (or the combine) merges."""
    run = gpu_cases.run_case("pass_32k", problems=[16], fused=fused)
    _properties(run)
    _compare(run, all_certified=True)
