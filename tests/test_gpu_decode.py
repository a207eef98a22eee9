"""GPU parity of kv_decode_attention (attention of a generated token over the compacted cache)
against the oracle, on seeded synthetic caches and on the cache the eviction pass compacts.

Tolerance: the kernel forms logits, the softmax and the weighted sum in fp32.  A logit of a d = 128
dot product carries an error of a few fp32 ulps of sum |q_i k_i| (about 1e-6 here), which moves each
softmax weight by about that fraction; the output, a convex combination of value rows, moves by at
most that times max |v|.  The test allows 2e-5 max|v| + 1e-5 |o|.
"""
import numpy as np
import pytest

from oracle import decode, evict
from paper_2609_30738_amd import _lib, api, workloads
from tests import gpu_cases

pytestmark = pytest.mark.gpu


def _dev(x):
    return api.to_device(np.ascontiguousarray(x))


def _check_out(out, di, k_host, v_host, lens, append, where):
    """Compare every (problem, head) output with the oracle over the rows in use."""
    o = out.reshape(len(lens), di.h_q, di.d)
    for p, L in enumerate(lens):
        kd = evict.decode(k_host[p, :, :L], di.dtype)
        vd = evict.decode(v_host[p, :, :L], di.dtype)
        qd = evict.decode(di.q[p], di.dtype)
        kn = evict.decode(di.k_new[p], di.dtype) if append else None
        vn = evict.decode(di.v_new[p], di.dtype) if append else None
        ref = decode.decode_attention(qd, kd, vd, di.scale, kn, vn)
        vmax = max(np.abs(vd).max() if L else 0.0, np.abs(vn).max() if append else 0.0)
        err = np.abs(o[p] - ref)
        bound = 2e-5 * vmax + 1e-5 * np.abs(ref)
        assert np.all(err <= bound), (f"{where} p={p} L={L}: worst error {err.max():.3g} at "
                                      f"{np.unravel_index(np.argmax(err - bound), err.shape)}")


def _run(di, append=True, where=""):
    import torch
    print(f"[gpu case] decode {where} dtype={di.dtype} h_q={di.h_q} h_kv={di.h_kv} d={di.d} "
          f"stride={di.row_stride} lens={list(di.lens)} append={append}", flush=True)
    cb = _lib.CacheBatch(di.dtype, di.h_q, di.h_kv, di.d, di.row_stride, di.lens)
    k, v = _dev(di.k), _dev(di.v)
    out = torch.empty(len(di.lens) * di.h_q * di.d, dtype=torch.float32, device="cuda")
    ws = torch.empty(max(_lib.decode_workspace_bytes(cb), 256), dtype=torch.uint8, device="cuda")
    _lib.decode_attention(cb, _dev(di.q), k, v, _dev(di.k_new) if append else None,
                          _dev(di.v_new) if append else None, di.scale, out, ws)
    torch.cuda.synchronize()
    return out.cpu().numpy(), api.to_host_bits(k), api.to_host_bits(v)


@pytest.mark.parametrize("dtype,d,h_q,h_kv", [("bf16", 128, 32, 8), ("bf16", 64, 8, 4),
                                              ("f32", 128, 4, 4), ("f32", 64, 16, 2),
                                              ("bf16", 128, 12, 4)])
@pytest.mark.parametrize("append", [True, False])
def test_decode_matches_oracle(dtype, d, h_q, h_kv, append):
    """Group sizes 1, 2, 3 (padded to 4), 4 and 8; lengths 1 .. 300 in one batch, including rows
    that leave a partial pass and a partial unrolled block."""
    lens = [1, 7, 96, 300, 130, 65]
    di = workloads.draw_decode(dtype, h_q, h_kv, d, 320, lens, seed=3)
    out, k_after, v_after = _run(di, append, "shapes")
    _check_out(out, di, di.k, di.v, lens, append, f"{dtype} d={d} G={h_q // h_kv}")
    if append:
        for p, L in enumerate(lens):  # row L now holds the new token; nothing else changed
            np.testing.assert_array_equal(k_after[p, :, L], di.k_new[p])
            np.testing.assert_array_equal(v_after[p, :, L], di.v_new[p])
            np.testing.assert_array_equal(np.delete(k_after[p], L, axis=1), np.delete(di.k[p], L, axis=1))
            np.testing.assert_array_equal(np.delete(v_after[p], L, axis=1), np.delete(di.v[p], L, axis=1))
    else:
        np.testing.assert_array_equal(k_after, di.k)
        np.testing.assert_array_equal(v_after, di.v)


def test_decode_generation_steps_append_in_place():
    """Four generated tokens in a row over the same cache buffers: each call appends its row and
    the next call attends to it from the cache."""
    import torch
    lens = [96, 40, 250]
    first = workloads.draw_decode("bf16", 32, 8, 128, 260, lens, seed=10)
    cb = _lib.CacheBatch("bf16", 32, 8, 128, 260, lens)
    k, v = _dev(first.k), _dev(first.v)
    k_ref, v_ref = first.k.copy(), first.v.copy()
    out = torch.empty(len(lens) * 32 * 128, dtype=torch.float32, device="cuda")
    ws = torch.empty(max(_lib.decode_workspace_bytes(cb), 256), dtype=torch.uint8, device="cuda")
    for step in range(4):
        di = workloads.draw_decode("bf16", 32, 8, 128, 260, lens, seed=100 + step)
        cur = [int(x) for x in cb.lens_host]
        print(f"[gpu case] decode step {step} lens={cur}", flush=True)
        _lib.decode_attention(cb, _dev(di.q), k, v, _dev(di.k_new), _dev(di.v_new), di.scale, out,
                              ws)
        torch.cuda.synchronize()
        _check_out(out.cpu().numpy(), di, k_ref, v_ref, cur, True, f"step {step}")
        for p, L in enumerate(cur):
            k_ref[p, :, L] = di.k_new[p]
            v_ref[p, :, L] = di.v_new[p]
        cb.advance()
    np.testing.assert_array_equal(api.to_host_bits(k), k_ref)
    np.testing.assert_array_equal(api.to_host_bits(v), v_ref)


def test_decode_long_cache_splits_rows():
    """An uncompacted 20000-row cache next to a 777-row one (few units: the rows are split over
    workgroups and the partials merged)."""
    lens = [20000, 777]
    di = workloads.draw_decode("bf16", 32, 8, 128, 20001, lens, seed=5)
    cb = _lib.CacheBatch("bf16", 32, 8, 128, 20001, lens)
    assert _lib.decode_workspace_bytes(cb) > 0
    out, _, _ = _run(di, True, "long")
    _check_out(out, di, di.k, di.v, lens, True, "long")


def test_decode_over_the_compacted_cache_of_the_pass():
    """Eviction pass on the GPU (one Mistral layer, L = 3000, B = 64), compaction into blocks with
    room for generated rows, then one decode step; compared with the oracle's compacted rows and
    decode attention for every kv head whose admissions equal the oracle's."""
    import torch
    wl = workloads.mistral_layer()
    wl.seq_lens = [3000]
    pk = workloads.draw_packed(wl)
    lam1, lam2 = gpu_cases.layer_lambdas(wl, [0])
    inp = api.upload(wl.dtype, wl.h_q, wl.h_kv, wl.d, wl.w, pk.q_win, pk.k, pk.v, pk.lens,
                     pk.tok_off, lam1, lam2)
    out = api.allocate(inp, wl.budget)
    print("[gpu case] decode after the eviction pass L=3000", flush=True)
    api.run_pass(inp, out, wl.budget)
    stride = wl.budget + wl.w + 2
    kc = torch.empty(wl.h_kv * stride * wl.d, dtype=inp.k.dtype, device="cuda")
    vc = torch.empty_like(kc)
    _lib.compact_cache_ex(inp.batch, inp.k, inp.v, out.sel_idx, wl.budget, wl.w, None, kc, vc,
                          out_rows=stride)
    di = workloads.draw_decode("bf16", wl.h_q, wl.h_kv, wl.d, stride, [wl.budget + wl.w], seed=9)
    cb = _lib.CacheBatch("bf16", wl.h_q, wl.h_kv, wl.d, stride, [wl.budget + wl.w])
    o = torch.empty(wl.h_q * wl.d, dtype=torch.float32, device="cuda")
    _lib.decode_attention(cb, _dev(di.q), kc, vc, _dev(di.k_new), _dev(di.v_new), di.scale, o)
    torch.cuda.synchronize()
    sel = out.sel_idx.cpu().numpy().reshape(wl.h_kv, wl.budget)
    L = 3000
    k = pk.k.reshape(wl.h_kv, L, wl.d)
    v = pk.v.reshape(wl.h_kv, L, wl.d)
    res = evict.evict_problem(pk.q_win[0], k, v, wl.dtype, wl.scale, float(lam1[0]),
                              float(lam2[0]), wl.budget)
    o = o.cpu().numpy().reshape(wl.h_q, wl.d)
    G = wl.h_q // wl.h_kv
    same = 0
    for g in range(wl.h_kv):
        if set(sel[g].tolist()) != set(res.heads[g].trace.selected):
            continue  # a near-tie admitted another row: its cache differs legitimately
        same += 1
        kd = evict.decode(res.k_out[g][None], wl.dtype)
        vd = evict.decode(res.v_out[g][None], wl.dtype)
        ref = decode.decode_attention(evict.decode(di.q[0, g * G:(g + 1) * G], wl.dtype), kd, vd,
                                      di.scale, evict.decode(di.k_new[0, g:g + 1], wl.dtype),
                                      evict.decode(di.v_new[0, g:g + 1], wl.dtype))
        vmax = max(np.abs(vd).max(), np.abs(evict.decode(di.v_new[0, g], wl.dtype)).max())
        err = np.abs(o[g * G:(g + 1) * G] - ref)
        assert np.all(err <= 2e-5 * vmax + 1e-5 * np.abs(ref)), f"g={g}: {err.max():.3g}"
    assert same >= wl.h_kv - 1, f"only {same} kv heads admitted the oracle's rows"
