"""GPU parity at the full workload sizes, in the benchmark's launch configuration (every layer of
every sequence in one batch), checked against the oracle on sampled problems and kv heads.

Every output of the batch is also checked for properties that hold at any size: admitted
positions are distinct candidates, the candidate lists are ascending, sum_i mu_i = 1 per head, and
the compacted tail equals the last W rows.
"""
import numpy as np
import pytest

from paper_2609_30738_amd import workloads
from tests import gpu_cases

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


def _sampled(run, problems, heads):
    reports = []
    for j in problems:
        reports += gpu_cases.check_problem(run, j, heads)
    print("  ", gpu_cases.summarize(reports), flush=True)


def test_headline_32_layers_L32768():
    """32 layers x L=32768, W=32, B=64, quadratic lambda2 profile (the benchmark workload)."""
    run = gpu_cases.run_gpu(workloads.mistral_pass_32k(), fused=True)
    _properties(run)
    _sampled(run, [0, 13, 16, 31], [0, 5])


@pytest.mark.parametrize("budget", [32, 64, 128])
def test_32_layers_L8192_segments(budget):
    run = gpu_cases.run_gpu(workloads.mistral_pass_8k(budget), fused=True)
    _properties(run)
    _sampled(run, [0, 10, 11, 21, 22, 31], [2])


def test_ragged_8x32_both_terms():
    """8 sequences (L ~ U{2048..31744}) x 32 layers, B=128, lambda1=0.3, lambda2=-0.15."""
    run = gpu_cases.run_gpu(workloads.ragged_batch("both"), fused=True)
    _properties(run)
    _sampled(run, [0, 37, 100, 255], [3])


@pytest.mark.parametrize("pool", [1, 5])
def test_long_context_select_from_global_scores(pool):
    """L = 40000 > the 34816 candidate scores the selection stages in LDS: the score keys are
    re-formed from mu / sigma in HBM on every pass (and pooled there), 2 layers."""
    wl = workloads.mistral_layer()
    wl.seq_lens = [40000]
    wl.n_layers = 2
    run = gpu_cases.run_gpu(wl, fused=True, pool=pool)
    _properties(run)
    _sampled(run, [0, 1], [1, 6])


def test_32_layers_L8192_unfused_one_segment_per_unit():
    """kv_window_scores, then kv_mu_sigma from its row statistics, on the whole 32-layer batch:
    every unit is one segment, so the first pass writes the row statistics itself."""
    run = gpu_cases.run_gpu(workloads.mistral_pass_8k(64), fused=False)
    _properties(run)
    _sampled(run, [0, 15, 31], [1, 6])


@pytest.mark.parametrize("fused", [True, False])
def test_one_layer_of_the_32k_pass_alone(fused):
    """One layer of the L=32768 workload launched by itself, as in the per-layer schedule: 32
    segments of 1024 keys per unit, whose partials the second pass (or the combine) merges."""
    run = gpu_cases.run_gpu(workloads.mistral_pass_32k(), problems=[16], fused=fused)
    _properties(run)
    _sampled(run, [0], [0, 3, 7])
