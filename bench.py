"""Benchmark of one eviction pass over a whole batch on one MI355X.

A step is the full hot path over every layer of the workload: window row statistics, per-token
mean/dispersion and base score, the candidate cut, greedy selection and cache compaction, with
every input already resident in HBM.  The timed pass is kv_evict_pass: one launch in which each
(layer, kv head) unit's workgroup forms the row statistics and the unit's candidate set (reading
the keys once in full and revisiting only the tiles whose score bound reaches the candidate cut),
then runs the greedy on the candidates and compacts the kept rows.  Default workload: 32 layers of a Mistral-7B-shaped
cache (32 query / 8 kv heads, d=128, bf16), L=32768, W=32, B=64, quadratic lambda2 depth profile.

Before every timed step a 512 MiB buffer is read (outside the timed region) so that no part of
the 2 GiB key cache is served from the 256 MB last-level cache.  Each step is timed with HIP
events on the launch stream, per entry point and in total.  Further timed loops run, on the same
inputs, the other scoring routes (base scores through HBM; mu and sigma through HBM; the two
streaming passes as separate launches, so that each kernel's duration is measured live), the
selection options, a decode step, and the per-layer schedule (the scoring launched once per
layer, then one batched selection and compaction).  The roofline entry describes the kernel of
the timed pass (the dominant kernel; with the evict path the only one).  One JSON line is
printed.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, published
MFMA_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix peak, published
PATHS = ("evict", "candidates", "scored", "mu_sigma", "unfused")
WORKLOADS = ("mistral32_L32768_W32_B64", "mistral32_L8192_W32_B64", "mistral_layer_L4096_W32_B64")


def make_workload(name: str):
    from paper_2609_30738_amd import workloads as W
    if name == "mistral32_L32768_W32_B64":
        return W.mistral_pass_32k()
    if name == "mistral32_L8192_W32_B64":
        return W.mistral_pass_8k(64)
    if name == "mistral_layer_L4096_W32_B64":
        return W.mistral_layer()
    raise SystemExit(f"unknown workload {name}; choose from {WORKLOADS}")


def lambdas(wl):
    """Per-problem coefficients from the library's depth-profile entry point."""
    from paper_2609_30738_amd import _lib
    l1 = _lib.depth_profile(wl.lam1.family, wl.lam1.params, wl.n_layers)
    l2 = _lib.depth_profile(wl.lam2.family, wl.lam2.params, wl.n_layers)
    idx = [wl.layer_of(p) for p in range(wl.n_prob)]
    return l1[idx], l2[idx]


def algorithmic_bytes(wl) -> dict:
    """Bytes the method must move per pass: K once and Q_W once (scoring), the kept
    rows of K and V read and written (compaction) and the admitted indices.  One launch of the
    first scoring pass must read K and Q_W and write the row statistics (row_max, row_sum); one
    launch of the second reads K, Q_W and the row statistics and writes mu and sigma."""
    e = 2 if wl.dtype == "bf16" else 4
    lens = wl.lens.astype(np.int64)
    n = wl.n_prob
    keys = int(lens.sum()) * wl.h_kv * wl.d * e
    queries = n * wl.w * wl.h_q * wl.d * e
    kept = n * 2 * 2 * (wl.budget + wl.w) * wl.h_kv * wl.d * e
    idx = n * 4 * wl.budget * wl.h_kv
    row_stats = n * wl.h_q * wl.w * 2 * 4
    mu_sigma = int(lens.sum()) * wl.h_kv * 2 * 4
    return {"scoring": keys + queries, "total": keys + queries + kept + idx,
            "stats_pass": keys + queries + row_stats,
            "mu_sigma_pass": keys + queries + row_stats + mu_sigma}


def mfma_flops(wl) -> float:
    """Dense logits of one scoring pass: every window row against every key, d MACs each."""
    lens = wl.lens.astype(np.int64)
    return 2.0 * float(lens.sum()) * wl.h_q * wl.w * wl.d


# sources that define each profiled kernel: its traffic record stays valid while they are unchanged
KERNEL_SOURCES = {
    "window_prune": ("stream_prune.hip", "select_gram.h", "compact_rows.h", "stream_passes.h",
                     "stream_common.h", "common.h"),
    "window_stream": ("stream_window.hip", "stream_passes.h", "stream_common.h", "common.h"),
    "stats_stream": ("stream_stats.hip", "stream_passes.h", "stream_common.h", "common.h"),
    "mu_sigma_stream": ("stream_mu_sigma.hip", "stream_passes.h", "stream_common.h", "common.h"),
}


def _code_only(text: str) -> str:
    """Source text without // and /* */ comments and blank lines: what decides the kernel."""
    out, i, n = [], 0, len(text)
    while i < n:
        if text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
        elif text[i] == '"':  # string literals are kept whole
            j = i + 1
            while j < n and text[j] != '"':
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        else:
            out.append(text[i])
            i += 1
    return "\n".join(l.rstrip() for l in "".join(out).splitlines() if l.strip())


def source_sha(kernel: str) -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2609_30738_amd", "csrc")
    for f in KERNEL_SOURCES[kernel]:
        with open(os.path.join(csrc, f), encoding="utf-8") as fh:
            h.update(f.encode() + _code_only(fh.read()).encode())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it was taken on the
    current sources of the kernel (null otherwise)."""
    if kernel not in KERNEL_SOURCES:
        return None
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("source_sha") != source_sha(kernel):
        return None
    return rec.get("hbm_bytes_per_launch")


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:  # pragma: no cover
        pass
    return "unknown"


def cpu_baseline(wl, packed_layers, single_thread_layers: int) -> dict:
    """The CPU oracle, as it stands: the whole pass (every layer) with its BLAS on every host
    thread, then the first layers single-threaded, scaled to the pass."""
    from oracle import evict, profiles
    lam1 = profiles.layer_lambdas(wl.lam1.family, wl.lam1.params, wl.n_layers)
    lam2 = profiles.layer_lambdas(wl.lam2.family, wl.lam2.params, wl.n_layers)
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threadpool_limits = None
        threads = os.cpu_count() or 1

    def run(layers):
        t0 = time.perf_counter()
        for j, (q, k, v) in enumerate(layers):
            layer = wl.layer_of(j)
            evict.evict_problem(q, k, v, wl.dtype, wl.scale, lam1[layer], lam2[layer], wl.budget)
        return time.perf_counter() - t0

    full_s = run(packed_layers)
    line = {"value": round(full_s * 1e3, 1), "unit": "ms", "cores": int(threads),
            "kind": "oracle",
            "sample": f"the whole pass: all {len(packed_layers)} layers of {wl.name}, "
                      f"BLAS on {threads} threads",
            "host_cpus": os.cpu_count(), "cpu_model": cpu_model()}
    if single_thread_layers > 0 and threadpool_limits is not None:
        n1 = min(single_thread_layers, len(packed_layers))
        with threadpool_limits(1):
            one_s = run(packed_layers[:n1])
        line["single_thread"] = {"value": round(one_s / n1 * len(packed_layers) * 1e3, 1),
                                 "unit": "ms", "cores": 1,
                                 "sample": f"{n1} of {len(packed_layers)} layers ({one_s:.1f} s), "
                                           "scaled to the pass"}
    return line


def copy_probe(torch, mib: int) -> None:
    """A plain copy of known size: each launch reads and writes exactly mib MiB of HBM."""
    n = mib << 20
    src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": n, "launches": 3}), flush=True)


def per_mean_of(events, n):
    """Mean ms between consecutive events of each recorded step."""
    return np.array([[e[i].elapsed_time(e[i + 1]) for i in range(n)] for e in events]).mean(axis=0)


def config_passes(torch, args) -> None:
    """One JSON line per workload of the other configurations: the same batched pass
    (kv_evict_pass with the compaction), timed the same way (cache read-flushed before every step,
    HIP events), with its algorithmic bytes per second, and beside it the two calls it stands for
    (kv_window_candidates, then kv_mmr_select_candidates) and the scored route
    (kv_window_base_scores, kv_mmr_select_scored).  The ragged batch's
    three coefficient runs differ in lambda1 as well, so each is a pass of its own."""
    from paper_2609_30738_amd import _lib, api, workloads as W
    flush_buf = torch.ones(128 << 20, dtype=torch.float32, device="cuda")
    cases = [W.mistral_layer()] + [W.mistral_pass_8k(b) for b in (32, 64, 128)]
    ragged = [W.ragged_batch(r) for r in ("dispersion_only", "redundancy_only", "both")]
    stream = torch.cuda.current_stream()

    def run(wl, packed):
        inp = api.upload(wl.dtype, wl.h_q, wl.h_kv, wl.d, wl.w, packed.q_win, packed.k, packed.v,
                         packed.lens, packed.tok_off, *lambdas(wl))
        out = api.allocate(inp, wl.budget)
        b = inp.batch
        score = torch.empty_like(out.mu)
        wsb = _lib.base_scores_workspace_bytes(b)
        ws_sc = torch.empty(wsb, dtype=torch.uint8, device="cuda") if wsb else None
        wcb = _lib.candidates_workspace_bytes(b, wl.budget, 4, wl.w)
        ws_c = torch.empty(wcb, dtype=torch.uint8, device="cuda")

        def evict():
            _lib.evict_pass(b, inp.q_win, inp.k, inp.v, inp.scale, inp.lambda1, inp.lambda2,
                            wl.budget, 4, wl.w, out.row_max, out.row_sum, out.sel_idx, ws_c,
                            k_out=out.k_out, v_out=out.v_out)

        def cand():
            _lib.window_candidates(b, inp.q_win, inp.k, inp.scale, inp.lambda1, wl.budget, 4,
                                   wl.w, out.row_max, out.row_sum, ws_c)

        def cand_sel():
            _lib.mmr_select_candidates(b, ws_c, inp.k, inp.v, inp.lambda2, wl.budget, 4, wl.w,
                                       out.sel_idx, k_out=out.k_out, v_out=out.v_out)

        def scored():
            _lib.window_base_scores(b, inp.q_win, inp.k, inp.scale, inp.lambda1, out.row_max,
                                    out.row_sum, score, ws=ws_sc)

        def scored_sel():
            _lib.mmr_select_scored(b, score, inp.k, inp.v, inp.lambda2, wl.budget, 4, wl.w,
                                   out.sel_idx, k_out=out.k_out, v_out=out.v_out)
        res = []
        for calls in ((evict,), (cand, cand_sel), (scored, scored_sel)):
            rows = []
            for it in range(args.warmup + args.steps):
                flush_buf.amax()
                evs = [torch.cuda.Event(enable_timing=True) for _ in range(len(calls) + 1)]
                evs[0].record(stream)
                for i, fn in enumerate(calls):
                    fn()
                    evs[i + 1].record(stream)
                if it >= args.warmup:
                    rows.append(evs)
            torch.cuda.synchronize()
            res.append(per_mean_of(rows, len(calls)))
        return float(res[0][0]), res[1], float(res[2].sum()), algorithmic_bytes(wl)

    def entry(ms, two, scored_ms, ab):
        return {"ms_per_pass": round(ms, 4), "GBps": round(ab["total"] / (ms * 1e-3) / 1e9, 1),
                "two_calls_ms": {"kv_window_candidates": round(float(two[0]), 4),
                                 "kv_mmr_select_candidates (compacting)": round(float(two[1]), 4),
                                 "total": round(float(two.sum()), 4)},
                "scored_route_ms": round(scored_ms, 4)}

    for wl in cases:
        packed = W.draw_packed(wl)
        ms, two, scored_ms, ab = run(wl, packed)
        print(json.dumps({"config": wl.name, "algorithmic_bytes": ab["total"],
                          **entry(ms, two, scored_ms, ab)}), flush=True)
    packed = W.draw_packed(ragged[0])  # the three runs share their inputs
    per_run = {}
    for wl in ragged:
        ms, two, scored_ms, ab = run(wl, packed)
        per_run[wl.name.rsplit("_B128_", 1)[-1]] = entry(ms, two, scored_ms, ab)
    print(json.dumps({"config": ragged[0].name.replace("_dispersion_only", ""),
                      "total_tokens_per_layer": int(packed.lens.sum() // ragged[0].n_layers),
                      "algorithmic_bytes": ab["total"], "runs": per_run}), flush=True)


def main() -> None:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=20,
                    help="untimed steps first: the step time settles over the first 10-20 passes")
    ap.add_argument("--workload", default=WORKLOADS[0], choices=WORKLOADS)
    ap.add_argument("--cpu-baseline", type=int, default=1,
                    help="1: time the CPU oracle on the whole pass (all host threads) and on "
                         "--cpu-single-layers layers single-threaded; 0: skip")
    ap.add_argument("--cpu-single-layers", type=int, default=8,
                    help="layers of the single-threaded oracle sample")
    ap.add_argument("--settle-ms", type=float, default=30.0,
                    help="untimed passes before the warm-up: at least 20 and for at least this "
                         "long (0: none).  From idle the engine clock ramps up over the first "
                         "20-40 passes, so that a short warm-up leaves the first timed steps "
                         "slower than the rest")
    ap.add_argument("--flush", choices=("read", "write"), default="read",
                    help="how the last-level cache is emptied before each timed step")
    ap.add_argument("--path", choices=PATHS, default=PATHS[0],
                    help="the timed pass: evict = kv_evict_pass (one launch); candidates = "
                         "kv_window_candidates + kv_mmr_select_candidates; scored = kv_window_base_scores + "
                         "kv_mmr_select_scored (base scores through HBM); mu_sigma = "
                         "kv_window_mu_sigma + kv_mmr_select_compact (mu and sigma through HBM); "
                         "unfused = kv_window_scores + kv_mu_sigma, then kv_mmr_select_compact")
    ap.add_argument("--configs", action="store_true",
                    help="only time the pass on the other workloads (one layer, the 8k sweep over B, "
                         "the ragged batch), one JSON line each")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="only run a plain device copy of this many MiB three times (the known-size "
                         "kernel that scales the HBM byte counters) and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU; --gpus must be 1",
                          "n_gpus": args.gpus}))
        raise SystemExit(2)

    import torch
    from paper_2609_30738_amd import _lib, api, workloads
    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    torch.cuda.set_device(0)
    if args.copy_probe_mib > 0:
        copy_probe(torch, args.copy_probe_mib)
        return
    if args.configs:
        _lib.lib()
        config_passes(torch, args)
        return
    _lib.lib()  # fail loudly if the library is missing

    wl = make_workload(args.workload)
    t_gen = time.perf_counter()
    packed = workloads.draw_packed(wl)
    lam1, lam2 = lambdas(wl)
    inp = api.upload(wl.dtype, wl.h_q, wl.h_kv, wl.d, wl.w, packed.q_win, packed.k, packed.v,
                     packed.lens, packed.tok_off, lam1, lam2)
    out = api.allocate(inp, wl.budget)
    gen_s = time.perf_counter() - t_gen
    # evicts the key cache from the 256 MB last-level cache before every timed step: a read of
    # 512 MiB (a write would leave dirty lines whose write-back lands in the timed region)
    flush_buf = torch.ones(128 << 20, dtype=torch.float32, device="cuda")

    def flush():
        if args.flush == "write":
            flush_buf.fill_(1.0)
        else:
            flush_buf.amax()
    stream = torch.cuda.current_stream()
    b = inp.batch
    # the candidate lists of the timed pass, and the base score of every key for the scored route
    ws_c_bytes = _lib.candidates_workspace_bytes(b, wl.budget, 4, wl.w)
    if ws_c_bytes == 0:
        raise SystemExit("kv_candidates_workspace_bytes rejected the workload")
    ws_c = torch.empty(ws_c_bytes, dtype=torch.uint8, device="cuda")
    score = torch.empty_like(out.mu)
    ws_sc_bytes = _lib.base_scores_workspace_bytes(b)
    ws_sc = torch.empty(ws_sc_bytes, dtype=torch.uint8, device="cuda") if ws_sc_bytes else None
    mu_sigma_path = args.path in ("mu_sigma", "unfused")

    def evict_pass():
        _lib.evict_pass(b, inp.q_win, inp.k, inp.v, inp.scale, inp.lambda1, inp.lambda2,
                        wl.budget, 4, wl.w, out.row_max, out.row_sum, out.sel_idx, ws_c,
                        k_out=out.k_out, v_out=out.v_out)

    def cand_scoring():
        _lib.window_candidates(b, inp.q_win, inp.k, inp.scale, inp.lambda1, wl.budget, 4, wl.w,
                               out.row_max, out.row_sum, ws_c)

    def cand_select():
        _lib.mmr_select_candidates(b, ws_c, inp.k, inp.v, inp.lambda2, wl.budget, 4, wl.w,
                                   out.sel_idx, k_out=out.k_out, v_out=out.v_out)

    def scored_scoring():
        _lib.window_base_scores(b, inp.q_win, inp.k, inp.scale, inp.lambda1, out.row_max,
                                out.row_sum, score, ws=ws_sc)

    def scored_select():
        _lib.mmr_select_scored(b, score, inp.k, inp.v, inp.lambda2, wl.budget, 4, wl.w,
                               out.sel_idx, k_out=out.k_out, v_out=out.v_out)

    def ms_scoring():
        _lib.window_mu_sigma(b, inp.q_win, inp.k, inp.scale, out.row_max, out.row_sum, out.mu,
                             out.sigma, out.ws)

    def ms_select():
        _lib.mmr_select_compact(b, out.mu, out.sigma, inp.k, inp.v, inp.lambda1, inp.lambda2,
                                wl.budget, 4, wl.w, out.sel_idx, out.k_out, out.v_out, out.ws)

    def unfused_scoring():
        _lib.window_scores(b, inp.q_win, inp.k, inp.scale, out.row_max, out.row_sum, out.ws)
        _lib.mu_sigma(b, inp.q_win, inp.k, inp.scale, out.row_max, out.row_sum, out.mu, out.sigma)

    # each route: its entry points in order, (name, call); the breakdown times each call
    routes = {"evict": [("kv_evict_pass (compacting)", evict_pass)],
              "candidates": [("kv_window_candidates", cand_scoring),
                             ("kv_mmr_select_candidates (compacting)", cand_select)],
              "scored": [("kv_window_base_scores", scored_scoring),
                         ("kv_mmr_select_scored (compacting)", scored_select)],
              "mu_sigma": [("kv_window_mu_sigma", ms_scoring), ("kv_mmr_select_compact", ms_select)],
              "unfused": [("kv_window_scores + kv_mu_sigma", unfused_scoring),
                          ("kv_mmr_select_compact", ms_select)]}
    calls = routes[args.path]
    names = [n for n, _ in calls]

    def step(evs):
        evs[0].record(stream)
        for i, (_, fn) in enumerate(calls):
            fn()
            evs[i + 1].record(stream)

    def new_events():
        return [torch.cuda.Event(enable_timing=True) for _ in range(len(calls) + 1)]

    # settle phase (--settle-ms, 30 ms by default; reported as "settle"): from idle the engine
    # clock ramps up over the first 20-40 passes, which a warm-up of a few steps does not cover
    settle_passes, t_settle = 0, time.perf_counter()
    while args.settle_ms > 0 and (settle_passes < 20 or
                                  (time.perf_counter() - t_settle) * 1e3 < args.settle_ms):
        flush()
        step(new_events())
        settle_passes += 1
        if settle_passes % 10 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    settle_ms = (time.perf_counter() - t_settle) * 1e3
    for _ in range(args.warmup):
        flush()
        step(new_events())
    torch.cuda.synchronize()
    print(f"# inputs drawn and uploaded in {gen_s:.1f} s; settled ({settle_passes} passes, "
          f"{settle_ms:.0f} ms) and warmed up", file=sys.stderr, flush=True)

    all_events = []
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    for _ in range(args.steps):
        flush()  # outside the events
        evs = new_events()
        step(evs)
        all_events.append(evs)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0

    def timed(*calls):
        """Mean ms of each call over `steps` iterations (after `warmup`), cache flushed before
        every iteration, HIP events between the calls on the launch stream."""
        rows_ = []
        for it in range(args.warmup + args.steps):
            flush()
            evs = [torch.cuda.Event(enable_timing=True) for _ in range(len(calls) + 1)]
            evs[0].record(stream)
            for c, fn in enumerate(calls):
                fn()
                evs[c + 1].record(stream)
            if it >= args.warmup:
                rows_.append(evs)
        torch.cuda.synchronize()
        t = np.array([[e[i].elapsed_time(e[i + 1]) for i in range(len(calls))] for e in rows_])
        return [float(x) for x in t.mean(axis=0)]

    # the other routes on the same inputs (the unfused one is covered by the per-kernel loop)
    other_routes = {}
    for name in ("evict", "candidates", "scored", "mu_sigma"):
        if name != args.path:
            t = timed(*[fn for _, fn in routes[name]])
            other_routes[name] = {n: round(x, 4) for (n, _), x in zip(routes[name], t)}
            other_routes[name]["total"] = round(sum(t), 4)
    # the candidates route's two launches, from the timed pass or from the loop above
    cand_ms = (list(per_mean_of(all_events, len(calls))) if args.path == "candidates"
               else [other_routes["candidates"][n] for n, _ in routes["candidates"]])

    # per kernel: the two scoring passes through their own entry points, events between them
    # (warm-up first: a kernel's first launch also loads its code); with one segment per unit,
    # kv_window_scores is the first pass alone, which writes the row statistics itself
    k_stats, k_mu = timed(
        lambda: _lib.window_scores(b, inp.q_win, inp.k, inp.scale, out.row_max, out.row_sum,
                                   out.ws),
        lambda: _lib.mu_sigma(b, inp.q_win, inp.k, inp.scale, out.row_max, out.row_sum, out.mu,
                              out.sigma))
    # selection and compaction as their two entry points (the timed pass runs them in one launch)
    k_sel, k_cmp = timed(
        lambda: _lib.mmr_select(b, out.mu, out.sigma, inp.k, inp.lambda1, inp.lambda2, wl.budget,
                                4, wl.w, out.sel_idx, None, None, None, out.ws),
        lambda: _lib.compact_cache(b, inp.k, inp.v, out.sel_idx, wl.budget, wl.w, out.k_out,
                                   out.v_out))

    # scoring options on the same workload: dispersion over all (head, row) values, a max-pooled
    # base score, the mean-free score
    # depth-decreasing budgets at the same total (B = 64 per layer on average, beta = 20): the
    # rows are strided by the largest budget
    sched = _lib.pyramid_budgets(wl.budget, wl.n_layers, 20.0)
    pyr = _lib.Budgets([int(sched[wl.layer_of(p)]) for p in range(wl.n_prob)])
    b_max = pyr.max
    sel_pyr = torch.empty(wl.n_prob * wl.h_kv * b_max, dtype=torch.int32, device="cuda")
    kv_rows = wl.n_prob * wl.h_kv * (b_max + wl.w) * wl.d
    k_pyr = torch.empty(kv_rows, dtype=inp.k.dtype, device="cuda")
    v_pyr = torch.empty(kv_rows, dtype=inp.v.dtype, device="cuda")
    v_pyr_sel, v_pyr_cmp = timed(
        lambda: _lib.mmr_select_ex(b, out.mu, out.sigma, inp.k, inp.lambda1, inp.lambda2, b_max, 4,
                                   wl.w, sel_pyr, ws=out.ws, budgets=pyr),
        lambda: _lib.compact_cache_ex(b, inp.k, inp.v, sel_pyr, b_max, wl.w, pyr, k_pyr, v_pyr))

    # generation after eviction: one decode step (one token per layer, every query head) over the
    # compacted B + W rows, and for contrast over the uncompacted L rows of the same layers
    # (the attention the eviction saves on every generated token)
    q_dec = torch.randn(wl.n_prob * wl.h_q * wl.d, device="cuda").to(inp.k.dtype)
    o_dec = torch.empty(wl.n_prob * wl.h_q * wl.d, dtype=torch.float32, device="cuda")
    cb_kept = _lib.CacheBatch(wl.dtype, wl.h_q, wl.h_kv, wl.d, wl.budget + wl.w,
                              [wl.budget + wl.w] * wl.n_prob)
    uniform = bool(np.all(packed.lens == packed.lens[0]))
    cb_full = _lib.CacheBatch(wl.dtype, wl.h_q, wl.h_kv, wl.d, int(packed.lens[0]),
                              [int(packed.lens[0])] * wl.n_prob) if uniform else None

    def dec_ws(cb):
        nb = _lib.decode_workspace_bytes(cb)
        return torch.empty(max(nb, 256), dtype=torch.uint8, device="cuda") if nb else None
    ws_kept = dec_ws(cb_kept)
    ws_full = dec_ws(cb_full) if uniform else None
    dec_calls = [lambda: _lib.decode_attention(cb_kept, q_dec, out.k_out, out.v_out, None, None,
                                               inp.scale, o_dec, ws_kept)]
    if uniform:
        dec_calls.append(lambda: _lib.decode_attention(cb_full, q_dec, inp.k, inp.v, None, None,
                                                       inp.scale, o_dec, ws_full))
    v_dec = timed(*dec_calls)

    v_all, v_pool, v_free = timed(
        lambda: _lib.window_mu_sigma_ex(b, inp.q_win, inp.k, inp.scale, "all_rows", out.row_max,
                                        out.row_sum, out.mu, out.sigma, out.ws),
        lambda: _lib.mmr_select_ex(b, out.mu, out.sigma, inp.k, inp.lambda1, inp.lambda2,
                                   wl.budget, 4, wl.w, out.sel_idx, ws=out.ws, pool=7),
        lambda: _lib.mmr_select_ex(b, out.mu, out.sigma, inp.k, inp.lambda1, inp.lambda2,
                                   wl.budget, 4, wl.w, out.sel_idx, ws=out.ws, w_mu=0.0))

    # the per-layer schedule: the scoring launched layer by layer (as a model would after each
    # layer's prefill, into the same output buffers), then one batched selection and compaction
    layer_batches = [_lib.Batch(wl.dtype, wl.h_q, wl.h_kv, wl.d, wl.w, [int(b.lens_host[p])],
                                [int(b.tok_off_host[p])]) for p in range(b.n_prob)]
    rows = wl.h_q * wl.w
    ws_lay_bytes = max(_lib.base_scores_workspace_bytes(lb) for lb in layer_batches)
    ws_lay = torch.empty(max(ws_lay_bytes, 256), dtype=torch.uint8, device="cuda")

    def layered_step(evs):
        evs[0].record(stream)
        for p, lb in enumerate(layer_batches):
            if mu_sigma_path:
                _lib.window_mu_sigma(lb, inp.q_win[p], inp.k, inp.scale,
                                     out.row_max[p * rows:(p + 1) * rows],
                                     out.row_sum[p * rows:(p + 1) * rows], out.mu, out.sigma,
                                     out.ws)
            else:
                _lib.window_base_scores(lb, inp.q_win[p], inp.k, inp.scale, inp.lambda1[p:p + 1],
                                        out.row_max[p * rows:(p + 1) * rows],
                                        out.row_sum[p * rows:(p + 1) * rows], score, ws=ws_lay)
        evs[1].record(stream)
        if mu_sigma_path:
            ms_select()
        else:
            scored_select()
        evs[2].record(stream)

    layer_events = []
    for it in range(args.warmup + args.steps):
        flush()
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        layered_step(evs)
        if it >= args.warmup:
            layer_events.append(evs)
    torch.cuda.synchronize()
    lay = np.array([[e[i].elapsed_time(e[i + 1]) for i in range(2)] for e in layer_events])
    lay_score, lay_rest = (float(x) for x in lay.mean(axis=0))

    per = np.array([[e[i].elapsed_time(e[i + 1]) for i in range(len(calls))] for e in all_events])
    step_ms = per.sum(axis=1)
    ms = float(step_ms.mean())
    mean_part = per.mean(axis=0)
    ab = algorithmic_bytes(wl)
    flops = mfma_flops(wl)
    # The dominant kernel is the first kernel of the timed pass: with the evict path the one launch
    # of window_prune_kernel that scores, cuts, selects and compacts (what the method must move
    # for it: K and Q_W once, the kept rows of K and V read and written, the indices), otherwise
    # the scoring kernel (K and Q_W once).  Its revisits of K and its workspace traffic are
    # overhead of the design and show in `traffic`.  roofline_passes gives the same view of the two
    # streaming passes run as separate launches.
    def roofline(kernel, alg, kms):
        achieved = alg / (kms * 1e-3) / 1e9
        return {"kernel": kernel, "bound": "hbm", "achieved": round(achieved, 1),
                "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": measured_traffic(kernel, wl.name),
                "algorithmic_bytes_per_launch": alg, "ms_per_launch": round(kms, 4)}
    dominant_kernel = {"evict": "window_prune", "candidates": "window_prune",
                       "scored": "window_stream", "mu_sigma": "window_stream",
                       "unfused": "stats_stream+mu_sigma_stream"}[args.path]
    dominant = roofline(dominant_kernel, ab["total"] if args.path == "evict" else ab["scoring"],
                        float(mean_part[0]))
    passes = [roofline("stats_stream", ab["scoring"], k_stats),
              roofline("mu_sigma_stream", ab["scoring"], k_mu)]
    line = {
        "metric": "ms per 32-layer eviction pass at L=32k,W=32,B=64; HBM GB/s vs peak",
        "value": round(ms, 4),
        "unit": "ms",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic (seeded; Mistral-7B-shaped cache, planted sink, near-duplicate "
                "clusters and repeated passages)",
        "config": {"workload": wl.name, "layers": wl.n_layers, "L": int(wl.seq_lens[0]),
                   "W": wl.w, "B": wl.budget, "h_q": wl.h_q, "h_kv": wl.h_kv, "d": wl.d,
                   "lambda2_profile": wl.lam2.family, "parallelism": "single GPU"},
        "pass_GBps": round(ab["total"] / (ms * 1e-3) / 1e9, 1),
        "pass_frac_of_hbm_peak": round(ab["total"] / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "breakdown_ms": {n: round(float(v), 4) for n, v in zip(names, mean_part)},
        "step_ms_min_max": [round(float(step_ms.min()), 4), round(float(step_ms.max()), 4)],
        "step_ms_median": round(float(np.median(step_ms)), 4),
        "step_ms_each": [round(float(x), 4) for x in step_ms],
        "wall_s_timed_loop": round(wall, 3),
        "cache_flush": f"{args.flush} of 512 MiB before every timed step",
        "settle": {"passes": settle_passes, "ms": round(settle_ms, 1)},
        "pass": ", ".join(names),
        "other_routes_ms": other_routes,
        "per_layer_schedule_ms": {"total": round(lay_score + lay_rest, 4),
                                  ("scoring (32 launches of kv_window_mu_sigma)" if mu_sigma_path
                                   else "scoring (32 launches of kv_window_base_scores)"):
                                  round(lay_score, 4),
                                  "select+compact (batched)": round(lay_rest, 4)},
        "per_kernel_ms": {f"{dominant_kernel} ({names[0]})": round(float(mean_part[0]), 4),
                          "window_prune (kv_window_candidates)": round(cand_ms[0], 4),
                          "stats_stream (kv_window_scores)": round(k_stats, 4),
                          "mu_sigma_stream (kv_mu_sigma)": round(k_mu, 4),
                          "mmr_select (kv_mmr_select_candidates (compacting))": round(cand_ms[1], 4),
                          "mmr_select (kv_mmr_select)": round(k_sel, 4),
                          "compact (kv_compact_cache)": round(k_cmp, 4)},
        "options_ms": {"kv_window_mu_sigma_ex (sigma over all G*W rows)": round(v_all, 4),
                       "kv_mmr_select_ex (pool 7)": round(v_pool, 4),
                       "kv_mmr_select_ex (w_mu 0)": round(v_free, 4),
                       "kv_mmr_select_ex (depth-decreasing budgets, beta 20, "
                       f"{int(sched[0])}..{int(sched[-1])})": round(v_pyr_sel, 4),
                       "kv_compact_cache_ex (same budgets)": round(v_pyr_cmp, 4)},
        "decode_step_ms": {f"over the compacted cache ({wl.budget + wl.w} rows per kv head)":
                           round(v_dec[0], 4),
                           f"over the full cache ({int(packed.lens[0])} rows per kv head)":
                           round(v_dec[1], 4) if uniform else None},
        "mfma_tflops": {"stats_stream": round(flops / (k_stats * 1e-3) / 1e12, 1),
                        "mu_sigma_stream": round(flops / (k_mu * 1e-3) / 1e12, 1),
                        "peak_bf16_dense": MFMA_PEAK_TFLOPS},
        "roofline": dominant,
        "roofline_passes": passes,
    }
    # the device work is complete and its buffers released before the host-side baseline (and
    # before the interpreter exits: no device memory or event outlives the run)
    torch.cuda.synchronize()
    del all_events, layer_events
    inp = out = score = ws_sc = ws_lay = ws_c = None
    torch.cuda.empty_cache()
    if args.cpu_baseline:
        layers = []
        for j in range(wl.n_prob):
            L = int(packed.lens[j])
            off = int(packed.tok_off[j]) * wl.h_kv * wl.d
            n = L * wl.h_kv * wl.d
            layers.append((packed.q_win[j], packed.k[off:off + n].reshape(wl.h_kv, L, wl.d),
                           packed.v[off:off + n].reshape(wl.h_kv, L, wl.d)))
        line["cpu_baseline"] = cpu_baseline(wl, layers, args.cpu_single_layers)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
