"""GPU parity: every C-ABI entry point against the CPU oracle on seeded synthetic inputs.

Sizes span several key chunks and MFMA tiles with ragged tails; the full-size workloads run in the
benchmark's launch configuration (all layers in one batch) and are checked on sampled problems.
"""
import numpy as np
import pytest

from paper_2609_30738_amd import _lib, workloads
from tests import gpu_cases

pytestmark = pytest.mark.gpu


def _all(run, heads=None, certified=False):
    """Compare every problem of a run with the oracle; certified=True: every head's inputs are
    margin-certified, so every head must reproduce the oracle exactly."""
    reports = gpu_cases.check_all(run, heads=heads)
    print("  ", gpu_cases.summarize(reports), flush=True)
    if certified:
        assert all(r.certified for r in reports), gpu_cases.summarize(reports)
        assert all(r.identical_steps == r.steps for r in reports)
    return reports


def test_tiny_f32_unfused_with_attention():
    """fp32 path, 2 query heads on 1 kv head, d=64, W=8 (general window reduction); certified."""
    _all(gpu_cases.run_case("tiny_f32", want_attn=True), certified=True)


def test_tiny_f32_fused_exact_greedy_over_all_candidates():
    """cand_mult = 0: the greedy runs over every prefix position; certified."""
    _all(gpu_cases.run_case("tiny_f32_all_candidates", fused=True), certified=True)


@pytest.mark.parametrize("case", ["tiny_f32_no_tail", "tiny_f32_tail3"])
def test_tiny_f32_keep_tail(case):
    _all(gpu_cases.run_case(case), certified=True)


def test_mistral_layer_unfused():
    """One Mistral-7B layer, bf16, L=4096, W=32, B=64, lambda1=0.3, lambda2=-0.8; certified inputs,
    so every admission is the oracle's."""
    _all(gpu_cases.run_case("mistral_layer"), certified=True)


def test_mistral_layer_timed_calls():
    """The benchmark's calls (kv_window_mu_sigma, kv_mmr_select_compact) on certified inputs."""
    _all(gpu_cases.run_case("mistral_layer", timed=True), certified=True)


def test_exact_duplicate_keys_ties_to_lower_position():
    """Clusters of bitwise identical keys: exact ties at the candidate cut and in the greedy argmax
    are decided by the lower position on both sides (R10), through the default and the benchmark
    calls."""
    for timed in (False, True):
        _all(gpu_cases.run_case("exact_duplicates", fused=True, timed=timed), certified=True)


def test_nonfinite_inputs_keep_indices_valid():
    """NaN and Inf planted in keys and in window queries (results unspecified, R21): every call
    succeeds, and every selection is B distinct candidate positions."""
    wl = workloads.mistral_layer()
    wl.seq_lens = [3000]
    wl.n_seq = 1
    pk = workloads.draw_packed(wl)
    L, d, G = 3000, wl.d, wl.h_q // wl.h_kv
    k = pk.k.reshape(wl.h_kv, L, d)
    nan, inf, ninf = np.uint16(0x7FC0), np.uint16(0x7F80), np.uint16(0xFF80)
    k[0, 100] = nan                 # a NaN key row
    k[1, 200, :5] = inf             # a key with infinite entries
    k[2, 300:310] = ninf            # ten keys of -inf entries
    k[3, :, 7] = nan                # a NaN component in every key of a head
    pk.q_win[0, 5 * G, 3] = nan     # a NaN window query of kv head 5's group
    pk.q_win[0, 6 * G + 1, :] = inf  # an infinite window query of kv head 6's group
    for fused in (True, False):
        run = gpu_cases.run_gpu(wl, fused=fused, packed=pk)
        for timed in (False, True):
            if timed:
                run = gpu_cases.run_gpu(wl, packed=pk, timed=True)
            B = run.budget
            sel = run.host["sel_idx"].reshape(wl.h_kv, B)
            for g in range(wl.h_kv):
                s = sel[g]
                assert len(set(s.tolist())) == B, f"g={g}: repeated positions {s}"
                assert np.all((s >= 0) & (s < L - wl.w)), f"g={g}: out of range {s}"


def test_mistral_layer_fused_with_attention_short_context():
    """Ragged context (L=1337: partial chunk and partial tile) with the attention output."""
    wl = workloads.mistral_layer()
    wl.seq_lens = [1337]
    _all(gpu_cases.run_gpu(wl, want_attn=True))


@pytest.mark.parametrize("budget", [32, 64, 128])
def test_segments_profile_budget_sweep_scaled(budget):
    """Three-segment lambda2 over 3 layers (one per segment), L=2048, B in {32, 64, 128}."""
    _all(gpu_cases.run_case(f"segments_scaled_B{budget}", fused=True))


def test_curve_profile_scaled():
    """Quadratic lambda2 profile with passages repeated twice, 4 layers of L=6000; certified."""
    _all(gpu_cases.run_case("curve_scaled", fused=True), certified=True)


@pytest.mark.parametrize("run", ["dispersion_only", "redundancy_only", "both"])
def test_ragged_batch_scaled(run):
    """Three sequences of different lengths x 2 layers, B=128, the three term-ablation runs."""
    _all(gpu_cases.run_case(f"ragged_scaled_{run}", fused=True))


def _plant_rising_keys(wl, pk, plants):
    """Per kv group, keys along head 0's mean query direction (orthogonal to the other heads'
    mean directions) with window logits of about alpha nats at the given positions of problem 0."""
    from oracle import evict
    q = evict.decode(pk.q_win[0], wl.dtype).astype(np.float64)  # [h_q, w, d]
    L = int(pk.lens[0])
    G = wl.h_q // wl.h_kv
    k = pk.k[: wl.h_kv * L * wl.d].reshape(wl.h_kv, L, wl.d)
    for g in range(wl.h_kv):
        dirs = [q[g * G + h].mean(axis=0) for h in range(G)]
        u = dirs[0].copy()
        basis = []
        for v in dirs[1:]:
            for b_ in basis:
                v = v - (v @ b_) * b_
            basis.append(v / np.linalg.norm(v))
        for b_ in basis:
            u = u - (u @ b_) * b_
        u /= np.linalg.norm(u)
        nu = float((q[g * G] @ u).mean())
        for pos, alpha in plants:
            k[g, pos] = workloads.f32_to_bf16_bits((alpha / (wl.scale * nu) * u).astype(np.float32))


@pytest.mark.parametrize("fused", [True, False])
def test_rising_logits_move_the_running_offset(fused):
    """Keys whose logits rise far above the earlier ones, in later tiles and segments of the unit:
    about 9 nats (kept against the running offset), 40 nats (a rebase) and 100 nats (2^x of the
    difference overflows; a rebase).  Row statistics, mu and sigma must still match."""
    wl = workloads.mistral_layer()
    wl.seq_lens = [5000]
    pk = workloads.draw_packed(wl)
    _plant_rising_keys(wl, pk, [(777, 9.0), (2222, 40.0), (4444, 100.0)])
    _all(gpu_cases.run_gpu(wl, fused=fused, packed=pk))


@pytest.mark.parametrize("pool", [3, 7, 31])
def test_max_pooled_scores(pool):
    """kv_mmr_select_ex with a max-pool over positions (the window stops at the end of the
    candidate range): two ragged sequences x 2 layers, B=64."""
    wl = workloads.ragged_batch("both", n_seq=2, n_layers=2, len_range=(700, 3100))
    wl.budget = 64
    _all(gpu_cases.run_gpu(wl, fused=True, pool=pool))


def test_max_pooled_scores_across_pooling_chunks():
    """bf16 keys, L = 20000: the in-place pooling of the staged keys runs in three chunks of
    8192 positions, so windows straddle chunk ends (pool 31)."""
    wl = workloads.mistral_layer()
    wl.seq_lens = [20000]
    _all(gpu_cases.run_gpu(wl, fused=True, pool=31), heads=[0, 3, 7])


def test_max_pooled_scores_fp32_chunks():
    """fp32 keys (256 threads, chunks of 2048 positions), L = 5000, pool 9."""
    wl = workloads.tiny_f32()
    wl.seq_lens = [5000]
    _all(gpu_cases.run_gpu(wl, fused=True, pool=9))


def test_max_pooled_scores_fp32_keep_all():
    """fp32 keys (256-thread select), every position a candidate (keep_tail = 0) and pool 5."""
    _all(gpu_cases.run_gpu(workloads.tiny_f32(), fused=True, keep_tail=0, pool=5))


@pytest.mark.parametrize("case", ["mean_free_dispersion_only", "mean_free"])
def test_mean_free_score(case):
    """w_mu = 0: the score without the mean term (dispersion and redundancy only)."""
    _all(gpu_cases.run_case(case, fused=True))


def test_mean_free_max_pooled_unfused():
    """w_mu = 0.5 and pool 9 together, through the two-call scoring path."""
    wl = workloads.mistral_layer()
    wl.seq_lens = [3000]
    _all(gpu_cases.run_gpu(wl, fused=False, w_mu=0.5, pool=9))


@pytest.mark.parametrize("fused", [True, False])
def test_dispersion_over_all_group_rows(fused):
    """KV_SIGMA_ALL_ROWS, 4 query heads per kv head: streaming pass 2 (fused) and the generic
    w = 32 kernel with the attention output (unfused), L = 3000."""
    _all(gpu_cases.run_case("sigma_all_rows", fused=fused, want_attn=not fused), certified=True)


@pytest.mark.parametrize("sigma_rows", ["group_mean", "all_rows"])
def test_three_query_heads_per_kv_head(sigma_rows):
    """G = 3 (w = 32): 96 window rows in four 32-row blocks, the last one padding; generic
    kernels, both dispersion readings, L = 2100."""
    _all(gpu_cases.run_case(f"g3_{sigma_rows}", fused=True), certified=True)


def test_dispersion_over_all_group_rows_general_window():
    """KV_SIGMA_ALL_ROWS through the LDS reduction of other window sizes (fp32, G = 2, w = 8)."""
    _all(gpu_cases.run_gpu(workloads.tiny_f32(), fused=True, sigma_rows="all_rows"))


def test_depth_decreasing_budgets():
    """Per-problem budgets from the depth schedule (B = 64 over 4 layers, beta = 20: 125, 85, 43,
    3), two sequences x 4 layers of L = 3000 and 2200: ragged greedy lengths, candidate counts and
    compacted blocks, padded steps."""
    from oracle import budgets
    from tests import certified_cases
    sched = budgets.pyramid_budgets(64, 4, 20.0)
    assert sched == [125, 85, 43, 3]
    assert certified_cases.options("depth_budgets").budgets == tuple(sched * 2)
    _all(gpu_cases.run_case("depth_budgets", fused=True))


def test_depth_decreasing_budgets_fp32_with_options():
    """fp32 keys (256-thread select), budgets 40 and 16 in one batch, with pool 3 and w_mu 0.5."""
    wl = workloads.tiny_f32()
    wl.n_seq, wl.seq_lens = 2, [512, 700]
    _all(gpu_cases.run_gpu(wl, fused=True, budgets=[40, 16], pool=3, w_mu=0.5))


def test_compaction_of_oracle_selection():
    """kv_compact_cache fed with the oracle's admissions reproduces the oracle's compacted rows."""
    import torch
    from oracle import evict
    from paper_2609_30738_amd import _lib, api
    wl = workloads.mistral_layer()
    wl.seq_lens = [900]
    print(f"[gpu case] compaction {wl.name} L=900", flush=True)
    pk = workloads.draw_packed(wl)
    q, k, v = pk.q_win[0], pk.k.reshape(wl.h_kv, 900, wl.d), pk.v.reshape(wl.h_kv, 900, wl.d)
    res = evict.evict_problem(q, k, v, wl.dtype, wl.scale, 0.3, -0.8, wl.budget)
    sel = np.array([res.heads[g].trace.selected for g in range(wl.h_kv)], dtype=np.int32)
    inp = api.upload(wl.dtype, wl.h_q, wl.h_kv, wl.d, wl.w, pk.q_win, pk.k, pk.v, pk.lens,
                     pk.tok_off, [0.3], [-0.8])
    rows = wl.budget + wl.w
    k_out = torch.empty(wl.h_kv * rows * wl.d, dtype=inp.k.dtype, device=inp.k.device)
    v_out = torch.empty_like(k_out)
    _lib.compact_cache(inp.batch, inp.k, inp.v, api.to_device(sel.reshape(-1)), wl.budget, wl.w,
                       k_out, v_out)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(api.to_host_bits(k_out).reshape(res.k_out.shape), res.k_out)
    np.testing.assert_array_equal(api.to_host_bits(v_out).reshape(res.v_out.shape), res.v_out)


def test_deterministic_repeat():
    """Two runs on the same inputs give bitwise-identical outputs (no races in the reductions)."""
    wl = workloads.mistral_pass_32k(n_layers=2, L=5000, n_clusters=16, n_passages=4)
    a = gpu_cases.run_gpu(wl, fused=True)
    b = gpu_cases.run_gpu(wl, fused=True, packed=a.packed)
    for name in ("row_max", "row_sum", "mu", "sigma", "sel_idx", "sel_score", "cand_idx",
                 "cand_corr", "k_out", "v_out"):
        np.testing.assert_array_equal(a.host[name], b.host[name], err_msg=name)


@pytest.mark.parametrize("fused", [True, False])
def test_short_contexts_near_the_window(fused):
    """Contexts of 33, 64, 65, 95 and 287 keys in one bf16 batch with per-problem budgets: one
    candidate, partial tiles, the causal triangle of the window across two tiles, tiles with no
    unmasked key for some rows."""
    wl = workloads.Workload(
        "short_contexts_W32", 1, workloads.BF16, 32, 8, 128, 32, 64, 5, 1, [33, 64, 65, 95, 287],
        workloads.Layout(cluster_density=0.02),
        workloads.ProfileSpec(workloads.PROFILE_GLOBAL, (float(np.arcsinh(0.3)),)),
        workloads.ProfileSpec(workloads.PROFILE_GLOBAL, (float(np.arcsinh(-0.8)),)))
    _all(gpu_cases.run_gpu(wl, fused=fused, budgets=[1, 8, 8, 16, 64]))


def _one_segment_per_unit(wl) -> bool:
    """Whether the streaming plan gives every unit a single segment (both passes of a unit then
    run in one workgroup): about one segment per compute unit, 1024 keys at least, in whole
    256-key steps, never longer than the longest context."""
    total = int(wl.lens.astype(np.int64).sum()) * wl.h_kv
    seg = max(1024, -(-(-(-total // 256)) // 256) * 256)
    seg = min(seg, -(-int(wl.lens.max()) // 256) * 256)
    return seg >= int(wl.lens.max())


@pytest.mark.parametrize("sigma_rows", ["group_mean", "all_rows"])
def test_both_passes_in_one_workgroup_ragged(sigma_rows):
    """256 units of 1024, 1000, 700 and 513 keys (8 layers of 4 sequences): each unit is one
    segment, so the fused entry point runs pass 1, the normalisers and pass 2 of a unit in one
    workgroup; ragged tails, whole tiles and the window's causal triangle."""
    wl = workloads.Workload(
        "one_segment_units_W32", 1, workloads.BF16, 32, 8, 128, 32, 32, 4, 8, [1024, 1000, 700, 513],
        workloads.Layout(cluster_density=0.02),
        workloads.ProfileSpec(workloads.PROFILE_GLOBAL, (float(np.arcsinh(0.3)),)),
        workloads.ProfileSpec(workloads.PROFILE_GLOBAL, (float(np.arcsinh(-0.8)),)))
    assert wl.n_prob * wl.h_kv == 256 and _one_segment_per_unit(wl)
    _all(gpu_cases.run_gpu(wl, fused=True, sigma_rows=sigma_rows))


@pytest.mark.parametrize("sigma_rows", ["group_mean", "all_rows"])
def test_segments_computed_by_a_waiting_workgroup(sigma_rows, monkeypatch):
    """Units of 4096 keys in 4 segments (one Mistral-shaped layer): both passes run in one launch,
    and a workgroup that stops waiting for its unit's other segments computes their partials
    itself.  A poll limit of 0, set from the host, sends every workgroup down that path: the
    results match the oracle and are bit-identical to those of the default path."""
    wl = workloads.mistral_layer()
    monkeypatch.delenv("KVEVICT_SPIN_LIMIT", raising=False)
    ref = gpu_cases.run_gpu(wl, fused=True, sigma_rows=sigma_rows)
    monkeypatch.setenv("KVEVICT_SPIN_LIMIT", "0")
    run = gpu_cases.run_gpu(wl, fused=True, sigma_rows=sigma_rows)
    for name in ("row_max", "row_sum", "mu", "sigma", "sel_idx", "k_out", "v_out"):
        assert np.array_equal(run.host[name], ref.host[name]), name
    _all(run)


def _shape_workload(h_q, h_kv, d, n_seq, n_layers, lens, budget=16):
    return workloads.Workload(
        f"bf16_hq{h_q}_hkv{h_kv}_d{d}_W32", 1, workloads.BF16, h_q, h_kv, d, 32, budget, n_seq,
        n_layers, list(lens), workloads.Layout(cluster_density=0.02),
        workloads.ProfileSpec(workloads.PROFILE_GLOBAL, (float(np.arcsinh(0.3)),)),
        workloads.ProfileSpec(workloads.PROFILE_GLOBAL, (float(np.arcsinh(-0.8)),)))


STREAM_SHAPES = [(8, 8, 64), (16, 8, 128), (8, 2, 64), (16, 8, 64), (8, 8, 128)]


@pytest.mark.parametrize("h_q,h_kv,d", STREAM_SHAPES)
@pytest.mark.parametrize("fused", [True, False])
def test_stream_shapes_several_segments(h_q, h_kv, d, fused):
    """bf16, W = 32, every head layout and head size the streaming kernels take (G = 1, 2, 4;
    d = 64, 128), units of 3000 and 2100 keys in several segments: both passes in one launch
    (fused) or as the two entry points."""
    wl = _shape_workload(h_q, h_kv, d, 2, 2, [3000, 2100])
    _all(gpu_cases.run_gpu(wl, fused=fused))


@pytest.mark.parametrize("h_q,h_kv,d", STREAM_SHAPES)
def test_stream_shapes_one_segment_per_unit(h_q, h_kv, d):
    """The same layouts with 256 units of at most 1024 keys: each unit is one segment, so both
    passes of a unit run in one workgroup."""
    n_prob = 256 // h_kv
    wl = _shape_workload(h_q, h_kv, d, 2, n_prob // 2, [1024, 777])
    assert _one_segment_per_unit(wl)
    _all(gpu_cases.run_gpu(wl, fused=True))


def test_segments_merged_by_the_second_launch():
    """192 units of 5000 keys in two segments each: 384 workgroups do not fit the chip at once, so
    the fused entry point takes two launches, the second merging the first's segment partials
    from the workspace."""
    wl = _shape_workload(32, 8, 128, 3, 8, [5000, 5000, 5000], budget=32)
    total = int(wl.lens.sum()) * wl.h_kv
    seg = min(max(1024, -(-(-(-total // 256)) // 256) * 256), -(-int(wl.lens.max()) // 256) * 256)
    n_seg = -(-int(wl.lens.max()) // seg)
    assert n_seg == 2 and n_seg * wl.n_prob * wl.h_kv > 256
    _all(gpu_cases.run_gpu(wl, fused=True))


@pytest.mark.parametrize("h_q,h_kv,d", STREAM_SHAPES)
def test_stream_shapes_late_segments_computed_by_the_waiting_workgroup(h_q, h_kv, d, monkeypatch):
    """Every head layout and head size with a poll limit of 0: each workgroup computes the other
    segments' partials itself; the results are bit-identical to the default path's."""
    wl = _shape_workload(h_q, h_kv, d, 2, 2, [3000, 2100])
    monkeypatch.delenv("KVEVICT_SPIN_LIMIT", raising=False)
    ref = gpu_cases.run_gpu(wl, fused=True)
    monkeypatch.setenv("KVEVICT_SPIN_LIMIT", "0")
    run = gpu_cases.run_gpu(wl, fused=True)
    for name in ("row_max", "row_sum", "mu", "sigma", "sel_idx", "k_out", "v_out"):
        assert np.array_equal(run.host[name], ref.host[name]), name


@pytest.mark.parametrize("case", ["mistral_layer", "pass_8k_B128_scaled", "tiny_f32", "tiny_f32_no_tail"])
def test_select_and_compact_in_one_launch(case):
    """kv_mmr_select_compact: the admission sequence and the compacted rows are bit-identical to
    kv_mmr_select followed by kv_compact_cache on the same scores (256 and 512 candidates in
    bf16, fp32 keys with and without the kept tail)."""
    import torch
    from paper_2609_30738_amd import _lib, api
    tail = None
    if case == "mistral_layer":
        wl = workloads.mistral_layer()
    elif case == "pass_8k_B128_scaled":
        wl = workloads.mistral_pass_8k(budget=128, n_layers=3, L=4096)
    else:
        wl = workloads.tiny_f32()
        tail = 0 if case == "tiny_f32_no_tail" else None
    keep = wl.w if tail is None else tail
    print(f"[gpu case] select+compact {case}", flush=True)
    packed = workloads.draw_packed(wl)
    import bench
    lam1, lam2 = bench.lambdas(wl)
    inp = api.upload(wl.dtype, wl.h_q, wl.h_kv, wl.d, wl.w, packed.q_win, packed.k, packed.v,
                     packed.lens, packed.tok_off, lam1, lam2)
    out = api.allocate(inp, wl.budget, 4, keep)
    b = inp.batch
    _lib.window_mu_sigma(b, inp.q_win, inp.k, inp.scale, out.row_max, out.row_sum, out.mu,
                         out.sigma, out.ws)
    _lib.mmr_select(b, out.mu, out.sigma, inp.k, inp.lambda1, inp.lambda2, wl.budget, 4, keep,
                    out.sel_idx, None, None, None, out.ws)
    _lib.compact_cache(b, inp.k, inp.v, out.sel_idx, wl.budget, keep, out.k_out, out.v_out)
    sel2, k2, v2 = (torch.full_like(out.sel_idx, -7), torch.zeros_like(out.k_out),
                    torch.zeros_like(out.v_out))
    _lib.mmr_select_compact(b, out.mu, out.sigma, inp.k, inp.v, inp.lambda1, inp.lambda2,
                            wl.budget, 4, keep, sel2, k2, v2, out.ws)
    torch.cuda.synchronize()
    assert torch.equal(sel2, out.sel_idx)
    assert torch.equal(k2.view(torch.int16 if k2.element_size() == 2 else torch.int32),
                       out.k_out.view(torch.int16 if k2.element_size() == 2 else torch.int32))
    assert torch.equal(v2.view(torch.int16 if v2.element_size() == 2 else torch.int32),
                       out.v_out.view(torch.int16 if v2.element_size() == 2 else torch.int32))


# ------------------------------------------------------------------------------------------------
# The benchmark's calls (kv_window_base_scores, then kv_mmr_select_scored with the compaction) with
# every scoring option and on every window path: fp32 batches take mu / sigma through the
# workspace and the base-score kernel, units in several segments the one-launch cooperative kernel
# (or, when its grid does not fit, the two-launch path), whole-unit workgroups the fused kernel.
# Each run also checks the scores bit for bit against the mu / sigma path's (tests/gpu_cases.py).
# ------------------------------------------------------------------------------------------------

@pytest.mark.parametrize("case,certified", [
    ("tiny_f32", True), ("tiny_f32_tail3", True), ("sigma_all_rows", True),
    ("g3_group_mean", True), ("g3_all_rows", True), ("curve_scaled", True),
    ("mean_free", False), ("depth_budgets", False)])
def test_scored_calls_with_options(case, certified):
    _all(gpu_cases.run_case(case, timed=True), certified=certified)


def test_scored_calls_max_pooled():
    """Pooling in the selection from given scores."""
    wl = workloads.ragged_batch("both", n_seq=2, n_layers=2, len_range=(700, 3100))
    wl.budget = 64
    _all(gpu_cases.run_gpu(wl, pool=7, timed=True))


@pytest.mark.parametrize("h_q,h_kv,d", STREAM_SHAPES)
def test_scored_calls_stream_shapes(h_q, h_kv, d):
    """Every streaming head layout and head size, one segment per unit (scores formed in the fused
    kernel) and several (in the cooperative kernel)."""
    n_prob = 256 // h_kv
    one = _shape_workload(h_q, h_kv, d, 2, n_prob // 2, [1024, 777])
    assert _one_segment_per_unit(one)
    _all(gpu_cases.run_gpu(one, timed=True))
    _all(gpu_cases.run_gpu(_shape_workload(h_q, h_kv, d, 2, 2, [3000, 2100]), timed=True))


def test_scored_calls_late_segments_and_second_launch(monkeypatch):
    """Base scores from the cooperative kernel's waiting-workgroup path (poll limit 0) equal the
    default path's bit for bit; a batch whose cooperative grid does not fit the chip forms them
    from mu / sigma in the workspace."""
    wl = workloads.mistral_layer()
    monkeypatch.delenv("KVEVICT_SPIN_LIMIT", raising=False)
    ref = gpu_cases.run_gpu(wl, timed=True)
    monkeypatch.setenv("KVEVICT_SPIN_LIMIT", "0")
    run = gpu_cases.run_gpu(wl, timed=True)
    for name in ("row_max", "row_sum", "score", "sel_idx", "k_out", "v_out"):
        assert np.array_equal(run.host[name], ref.host[name]), name
    _all(run)
    monkeypatch.delenv("KVEVICT_SPIN_LIMIT", raising=False)
    big = _shape_workload(32, 8, 128, 3, 8, [5000, 5000, 5000], budget=32)
    _all(gpu_cases.run_gpu(big, timed=True))


@pytest.mark.parametrize("h_q,h_kv,d,lens,budget,cand_mult", [
    (8, 8, 64, [8192, 8161], 16, 4), (8, 8, 64, [8192, 8161], 37, 3),
    (8, 8, 64, [8192, 8161], 72, 4), (8, 8, 64, [8192, 8161], 128, 4),
    (32, 8, 128, [4096, 4065], 37, 3), (32, 8, 128, [4096, 4065], 96, 4)])
def test_candidates_cut_in_the_window_kernel(h_q, h_kv, d, lens, budget, cand_mult):
    """256 units of one segment each, 4065 to 8192 keys, 2 % planted keys, so that for C above
    their count the cut falls in the bulk: the candidate kernel codes every tile's row maxima in
    pass 1, bounds the
    tiles' scores once the normalisers are known, revisits tiles in decreasing order of their
    bounds until the cut passes them, and finds the C-th largest of the evaluated entries digit by
    digit (C = 64, 111, 288, 512 and 384).  The selection from its candidates equals
    kv_mmr_select_ex's, every output bit for bit, and the oracle's."""
    wl = _shape_workload(h_q, h_kv, d, 2, 16, lens, budget=budget)
    assert wl.n_prob * wl.h_kv == 256 and _one_segment_per_unit(wl)
    b = _lib.Batch(wl.dtype, h_q, h_kv, d, wl.w, wl.lens, device="cpu")
    C = cand_mult * budget
    lists = 256 * C * 8
    codes = 256 * ((max(lens) + 31) // 32) * 128  # 128 bytes per tile of the longest unit
    # the lists are formed in the window pass: the workspace holds them, the normalisers and the
    # first pass's tile codes only
    assert _lib.candidates_workspace_bytes(b, budget, cand_mult, wl.w) == lists + 1024 + codes
    run = gpu_cases.run_gpu(wl, cand_mult=cand_mult, timed=True)
    assert "cands_sel_idx" in run.host
    _all(run)
