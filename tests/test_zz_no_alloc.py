"""kv_window_mu_sigma_noalloc (the entry point that allocates nothing) against kv_window_mu_sigma
with a caller workspace, bit for bit, on two calls in a row, the second with a smaller batch.  The
batches take the paths that use scratch: one layer whose units span several segments (both passes
in one launch, arrival counters and partials in scratch) and a batch too large for one launch (the
second launch merges the partials from scratch)."""
import numpy as np
import pytest

from paper_2609_30738_amd import _lib, api, workloads

pytestmark = pytest.mark.gpu


def _layer(L, n_layers=1, n_seq=1):
    wl = workloads.mistral_layer()
    wl.seq_lens = [L] * n_seq
    wl.n_seq = n_seq
    wl.n_layers = n_layers
    return wl


@pytest.mark.parametrize("sigma_rows", ["group_mean", "all_rows"])
def test_no_alloc_entry_matches_the_workspace_entry(sigma_rows):
    import torch
    cases = [_layer(4096), _layer(3000),            # one launch, 4 then 3 segments per unit
             _layer(5000, n_layers=8, n_seq=3), _layer(2500, n_layers=8, n_seq=3)]  # two launches
    for wl in cases:
        print(f"[gpu case] no-alloc {wl.name} L={wl.seq_lens} problems={wl.n_prob} {sigma_rows}",
              flush=True)
        pk = workloads.draw_packed(wl)
        inp = api.upload(wl.dtype, wl.h_q, wl.h_kv, wl.d, wl.w, pk.q_win, pk.k, pk.v, pk.lens,
                         pk.tok_off, [0.3] * wl.n_prob, [-0.8] * wl.n_prob)
        ref = api.allocate(inp, wl.budget)
        got = api.allocate(inp, wl.budget)
        for t in (got.row_max, got.row_sum, got.mu, got.sigma):
            t.fill_(float("nan"))
        b = inp.batch
        assert _lib.workspace_bytes(b, wl.budget, 4, wl.w) > 256  # the path uses scratch
        _lib.window_mu_sigma_ex(b, inp.q_win, inp.k, inp.scale, sigma_rows, ref.row_max,
                                ref.row_sum, ref.mu, ref.sigma, ref.ws)
        _lib.window_mu_sigma_noalloc(b, inp.q_win, inp.k, inp.scale, got.row_max, got.row_sum,
                                     got.mu, got.sigma, sigma_rows)
        torch.cuda.synchronize()
        for name in ("row_max", "row_sum", "mu", "sigma"):
            a = api.to_host_bits(getattr(ref, name))
            g = api.to_host_bits(getattr(got, name))
            assert np.array_equal(a.view(np.uint32), g.view(np.uint32)), name
