"""Named parity cases whose inputs are margin-certified (see tests/certify.py).

Each case is a seeded workload plus the selection options the GPU runs it with.  The positions
that certification re-draws are stored in tests/golden/certified_inputs.json (written by
tests/golden/make_certified.py, which runs only the oracle); `inputs(name)` draws the case's inputs
with them applied.
"""
from __future__ import annotations

import json
import os
from typing import Callable, Dict, Optional, Tuple

import numpy as np

from paper_2609_30738_amd import workloads as W
from tests.certify import Options, Redraw

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "certified_inputs.json")


def _scaled_8k(budget):
    return lambda: W.mistral_pass_8k(budget=budget, n_layers=3, L=2048)


def _ragged_scaled(run):
    return lambda: W.ragged_batch(run, n_seq=3, n_layers=2, len_range=(700, 3100))


def _layer(L):
    def make():
        wl = W.mistral_layer()
        wl.seq_lens = [L]
        wl.name = f"mistral_layer_L{L}_W32_B64"
        return wl
    return make


def _budgets_case():
    wl = W.mistral_pass_8k(n_layers=4, L=3000)
    wl.n_seq, wl.seq_lens = 2, [3000, 2200]
    wl.name = "mistral4x2_L3000-2200_W32_B64"
    return wl


def _g3():
    wl = W.mistral_layer()
    wl.h_q, wl.h_kv = 12, 4
    wl.seq_lens = [2100]
    wl.name = "layer_12q_4kv_L2100_W32_B64"
    return wl


def _exact_duplicates():
    """Clusters of bitwise identical keys (no noise): exact ties at the candidate boundary and in
    the greedy argmax, decided by the lower position on both sides (R10)."""
    wl = W.Workload("exact_duplicates_L4096_W32_B64", 5, W.BF16, 32, 8, 128, 32, 64, 1, 2, [4096],
                    W.Layout(n_clusters=24, cluster_size=16, noise_rel=0.0),
                    W.ProfileSpec(W.PROFILE_GLOBAL, (float(np.arcsinh(0.3)),)),
                    W.ProfileSpec(W.PROFILE_GLOBAL, (float(np.arcsinh(-0.8)),)))
    return wl


# name -> (workload constructor, options)
CASES: Dict[str, Tuple[Callable[[], W.Workload], Options]] = {
    # the five configurations at full size
    "tiny_f32": (W.tiny_f32, Options()),
    "mistral_layer": (W.mistral_layer, Options()),
    "pass_8k_B32": (lambda: W.mistral_pass_8k(32), Options()),
    "pass_8k_B64": (lambda: W.mistral_pass_8k(64), Options()),
    "pass_8k_B128": (lambda: W.mistral_pass_8k(128), Options()),
    "pass_32k": (W.mistral_pass_32k, Options()),
    "ragged_dispersion_only": (lambda: W.ragged_batch("dispersion_only"), Options()),
    "ragged_redundancy_only": (lambda: W.ragged_batch("redundancy_only"), Options()),
    "ragged_both": (lambda: W.ragged_batch("both"), Options()),
    # scaled cases and options
    "tiny_f32_all_candidates": (W.tiny_f32, Options(cand_mult=0)),
    "tiny_f32_no_tail": (W.tiny_f32, Options(keep_tail=0)),
    "tiny_f32_tail3": (W.tiny_f32, Options(keep_tail=3)),
    "segments_scaled_B32": (_scaled_8k(32), Options()),
    "segments_scaled_B64": (_scaled_8k(64), Options()),
    "segments_scaled_B128": (_scaled_8k(128), Options()),
    "curve_scaled": (lambda: W.mistral_pass_32k(n_layers=4, L=6000, n_clusters=16, n_passages=4),
                     Options()),
    "ragged_scaled_dispersion_only": (_ragged_scaled("dispersion_only"), Options()),
    "ragged_scaled_redundancy_only": (_ragged_scaled("redundancy_only"), Options()),
    "ragged_scaled_both": (_ragged_scaled("both"), Options()),
    "mean_free": (_ragged_scaled("both"), Options(w_mu=0.0)),
    "mean_free_dispersion_only": (_ragged_scaled("dispersion_only"), Options(w_mu=0.0)),
    "sigma_all_rows": (_layer(3000), Options(sigma_all_rows=True)),
    "g3_group_mean": (_g3, Options()),
    "g3_all_rows": (_g3, Options(sigma_all_rows=True)),
    "depth_budgets": (_budgets_case, Options(budgets=(125, 85, 43, 3, 125, 85, 43, 3))),
    "exact_duplicates": (_exact_duplicates, Options()),
}


# cases whose certification covers only some problems (the ones the tests compare with the oracle):
# the ragged batch, every layer of sequences 1 (30053 keys) and 7 (4448 keys)
RAGGED_COMPARED_SEQS = (1, 7)
PROBLEMS = {f"ragged_{r}": [s * 32 + l for s in RAGGED_COMPARED_SEQS for l in range(32)]
            for r in ("dispersion_only", "redundancy_only", "both")}


def workload(name: str) -> W.Workload:
    return CASES[name][0]()


def problems(name: str) -> Optional[list]:
    """The problems a case certifies (None: all)."""
    return PROBLEMS.get(name)


def options(name: str) -> Options:
    return CASES[name][1]


def load_redraw(name: str) -> Redraw:
    """Stored positions to re-draw for a case (empty if the case needed none)."""
    with open(GOLDEN) as f:
        rec = json.load(f)["cases"]
    if name not in rec:
        raise KeyError(f"{name}: no certified inputs stored; run tests/golden/make_certified.py")
    return {int(p): {int(g): list(v) for g, v in d.items()} for p, d in rec[name]["redraw"].items()}


def inputs(name: str, problems: Optional[list] = None) -> Tuple[W.Workload, W.PackedInputs, Redraw]:
    wl = workload(name)
    red = load_redraw(name)
    return wl, W.draw_packed(wl, problems, redraw=red), red
