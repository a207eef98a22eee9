"""ctypes binding of libkvevict.so, with the same names as the C ABI (include/kvevict.h).

Argument marshalling only: every function checks that tensors are contiguous device tensors,
passes their addresses and the current HIP stream, and raises KvError on a negative status.  All
computation happens in the library's gfx950 kernels.  Loading fails loudly if the library has not
been built; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

KV_OK = 0
KV_ERR_NULL = -1
KV_ERR_SHAPE = -2
KV_ERR_DTYPE = -3
KV_ERR_BUDGET = -4
KV_ERR_WORKSPACE = -5
KV_ERR_LAUNCH = -6
KV_ERR_ARG = -7
KV_ERR_SCRATCH = -8
KV_NOALLOC_SCRATCH_BYTES = 16 << 20

KV_SIGMA_GROUP_MEAN = 0
KV_SIGMA_ALL_ROWS = 1
SIGMA_ROWS = {"group_mean": KV_SIGMA_GROUP_MEAN, "all_rows": KV_SIGMA_ALL_ROWS}

KV_F32 = 0
KV_BF16 = 1

KV_PROFILE_GLOBAL = 0
KV_PROFILE_SEGMENTS = 1
KV_PROFILE_CURVE = 2
PROFILE_FAMILIES = {"global": KV_PROFILE_GLOBAL, "segments": KV_PROFILE_SEGMENTS,
                    "curve": KV_PROFILE_CURVE}

# KVEVICT_LIB selects another build of the same library (the host-sanitized one of the CPU tests)
LIB_PATH = os.environ.get("KVEVICT_LIB") or os.path.join(os.path.dirname(os.path.abspath(__file__)),
                                                         "libkvevict.so")

SYMBOLS = ("kv_strerror", "kv_version", "kv_workspace_bytes", "kv_candidate_stride",
           "kv_window_scores", "kv_mu_sigma", "kv_mu_sigma_ex", "kv_window_mu_sigma",
           "kv_window_mu_sigma_ex", "kv_window_mu_sigma_noalloc", "kv_window_base_scores",
           "kv_base_scores_workspace_bytes", "kv_mmr_select", "kv_mmr_select_ex",
           "kv_mmr_select_compact", "kv_mmr_select_scored", "kv_window_candidates",
           "kv_candidates_workspace_bytes", "kv_mmr_select_candidates", "kv_evict_pass",
           "kv_compact_cache", "kv_compact_cache_ex", "kv_decode_workspace_bytes",
           "kv_decode_attention", "kv_pyramid_budgets", "kv_depth_profile")


class KvError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {strerror(status)} (status {status})")


class KvProblem(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int32), ("n_prob", ctypes.c_int32), ("h_q", ctypes.c_int32),
                ("h_kv", ctypes.c_int32), ("d", ctypes.c_int32), ("w", ctypes.c_int32),
                ("len_host", ctypes.c_void_p), ("tok_off_host", ctypes.c_void_p),
                ("len_dev", ctypes.c_void_p), ("tok_off_dev", ctypes.c_void_p)]


class KvCacheBatch(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int32), ("n_prob", ctypes.c_int32), ("h_q", ctypes.c_int32),
                ("h_kv", ctypes.c_int32), ("d", ctypes.c_int32), ("row_stride", ctypes.c_int32),
                ("len_host", ctypes.c_void_p), ("len_dev", ctypes.c_void_p)]


class KvSelectOpts(ctypes.Structure):
    _fields_ = [("pool", ctypes.c_int32), ("w_mu", ctypes.c_float),
                ("budget_host", ctypes.c_void_p), ("budget_dev", ctypes.c_void_p)]


_LIB = None


def lib() -> ctypes.CDLL:
    """The loaded library (raises if it has not been built)."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        h = ctypes.CDLL(LIB_PATH)
        vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        pr = ctypes.POINTER(KvProblem)
        h.kv_strerror.argtypes = [ctypes.c_int]
        h.kv_strerror.restype = ctypes.c_char_p
        h.kv_version.argtypes = []
        h.kv_version.restype = ctypes.c_int
        h.kv_workspace_bytes.argtypes = [pr, i32, i32, i32]
        h.kv_workspace_bytes.restype = sz
        h.kv_candidate_stride.argtypes = [pr, i32, i32, i32]
        h.kv_candidate_stride.restype = i32
        h.kv_window_scores.argtypes = [pr, vp, vp, ctypes.c_float, vp, vp, vp, sz, vp]
        h.kv_mu_sigma.argtypes = [pr, vp, vp, ctypes.c_float, vp, vp, vp, vp, vp, vp]
        h.kv_window_mu_sigma.argtypes = [pr, vp, vp, ctypes.c_float, vp, vp, vp, vp, vp, sz, vp]
        h.kv_mu_sigma_ex.argtypes = [pr, vp, vp, ctypes.c_float, vp, vp, i32, vp, vp, vp, vp]
        h.kv_window_mu_sigma_ex.argtypes = [pr, vp, vp, ctypes.c_float, i32, vp, vp, vp, vp, vp,
                                            sz, vp]
        h.kv_window_mu_sigma_noalloc.argtypes = [pr, vp, vp, ctypes.c_float, i32, vp, vp, vp, vp,
                                                 vp]
        h.kv_window_base_scores.argtypes = [pr, vp, vp, ctypes.c_float, vp, ctypes.c_float, i32,
                                            vp, vp, vp, vp, sz, vp]
        h.kv_base_scores_workspace_bytes.argtypes = [pr]
        h.kv_base_scores_workspace_bytes.restype = sz
        h.kv_mmr_select_scored.argtypes = [pr, vp, vp, vp, vp, i32, i32, i32,
                                           ctypes.POINTER(KvSelectOpts), vp, vp, vp, vp, vp, vp, vp]
        h.kv_window_candidates.argtypes = [pr, vp, vp, ctypes.c_float, vp, i32, i32, i32, i32,
                                           ctypes.POINTER(KvSelectOpts), vp, vp, vp, sz, vp]
        h.kv_candidates_workspace_bytes.argtypes = [pr, i32, i32, i32,
                                                    ctypes.POINTER(KvSelectOpts)]
        h.kv_candidates_workspace_bytes.restype = sz
        h.kv_mmr_select_candidates.argtypes = [pr, vp, sz, vp, vp, vp, i32, i32, i32,
                                               ctypes.POINTER(KvSelectOpts), vp, vp, vp, vp, vp,
                                               vp, vp]
        h.kv_evict_pass.argtypes = [pr, vp, vp, vp, ctypes.c_float, vp, vp, i32, i32, i32, i32,
                                    ctypes.POINTER(KvSelectOpts), vp, vp, vp, vp, vp, vp, vp, sz,
                                    vp]
        h.kv_mmr_select.argtypes = [pr, vp, vp, vp, vp, vp, i32, i32, i32, vp, vp, vp, vp, vp, sz,
                                    vp]
        h.kv_mmr_select_compact.argtypes = [pr, vp, vp, vp, vp, vp, vp, i32, i32, i32, vp, vp, vp,
                                            vp, sz, vp]
        h.kv_mmr_select_ex.argtypes = [pr, vp, vp, vp, vp, vp, i32, i32, i32,
                                       ctypes.POINTER(KvSelectOpts), vp, vp, vp, vp, vp, sz, vp]
        h.kv_compact_cache.argtypes = [pr, vp, vp, vp, i32, i32, vp, vp, vp]
        h.kv_compact_cache_ex.argtypes = [pr, vp, vp, vp, i32, i32, vp, vp, i32, vp, vp, vp]
        cb = ctypes.POINTER(KvCacheBatch)
        h.kv_decode_workspace_bytes.argtypes = [cb]
        h.kv_decode_workspace_bytes.restype = sz
        h.kv_decode_attention.argtypes = [cb, vp, vp, vp, vp, vp, ctypes.c_float, vp, vp, sz, vp]
        h.kv_pyramid_budgets.argtypes = [i32, i32, ctypes.c_double, ctypes.POINTER(ctypes.c_int32)]
        h.kv_depth_profile.argtypes = [i32, ctypes.POINTER(ctypes.c_double), i32, i32,
                                       ctypes.POINTER(ctypes.c_float)]
        for name in ("kv_window_scores", "kv_mu_sigma", "kv_mu_sigma_ex", "kv_window_mu_sigma",
                     "kv_window_mu_sigma_ex", "kv_window_mu_sigma_noalloc",
                     "kv_window_base_scores", "kv_mmr_select", "kv_mmr_select_ex",
                     "kv_mmr_select_scored", "kv_window_candidates", "kv_mmr_select_candidates",
                     "kv_evict_pass", "kv_compact_cache", "kv_compact_cache_ex", "kv_decode_attention",
                     "kv_pyramid_budgets", "kv_depth_profile"):
            getattr(h, name).restype = ctypes.c_int
        _LIB = h
    return _LIB


def strerror(status: int) -> str:
    return lib().kv_strerror(int(status)).decode()


def version() -> int:
    return int(lib().kv_version())


def _check(status: int, where: str) -> None:
    if status != KV_OK:
        raise KvError(status, where)


class Batch:
    """Shape of a batch of problems (one problem = one layer of one sequence).

    Holds the host lengths/offsets and their device copies and exposes the kv_problem struct.
    """

    def __init__(self, dtype: str, h_q: int, h_kv: int, d: int, w: int, lens: Sequence[int],
                 tok_off: Optional[Sequence[int]] = None, device=None):
        import torch
        self.dtype_name = dtype
        self.h_q, self.h_kv, self.d, self.w = int(h_q), int(h_kv), int(d), int(w)
        self.lens_host = np.ascontiguousarray(np.asarray(lens, dtype=np.int32))
        if tok_off is None:
            off = np.zeros(len(self.lens_host), dtype=np.int64)
            if len(off) > 1:
                off[1:] = np.cumsum(self.lens_host.astype(np.int64))[:-1]
        else:
            off = np.asarray(tok_off, dtype=np.int64)
        self.tok_off_host = np.ascontiguousarray(off)
        dev = torch.device("cuda") if device is None else torch.device(device)
        self.lens_dev = torch.from_numpy(self.lens_host).to(dev)
        self.tok_off_dev = torch.from_numpy(self.tok_off_host).to(dev)
        self.struct = KvProblem(KV_BF16 if dtype == "bf16" else KV_F32, len(self.lens_host),
                                self.h_q, self.h_kv, self.d, self.w,
                                self.lens_host.ctypes.data, self.tok_off_host.ctypes.data,
                                self.lens_dev.data_ptr(), self.tok_off_dev.data_ptr())

    @property
    def n_prob(self) -> int:
        return len(self.lens_host)

    @property
    def total_tokens(self) -> int:
        return int(self.lens_host.astype(np.int64).sum())

    def ref(self):
        return ctypes.byref(self.struct)


class Budgets:
    """Per-problem budgets B_p: the host values and their device copy (budget_host / budget_dev of
    kv_select_opts and kv_compact_cache_ex)."""

    def __init__(self, values: Sequence[int], device=None):
        import torch
        self.host = np.ascontiguousarray(np.asarray(values, dtype=np.int32))
        dev = torch.device("cuda") if device is None else torch.device(device)
        self.dev = torch.from_numpy(self.host).to(dev)

    @property
    def max(self) -> int:
        return int(self.host.max())

    def pointers(self):
        return ctypes.c_void_p(self.host.ctypes.data), ctypes.c_void_p(self.dev.data_ptr())


def _ptr(t) -> ctypes.c_void_p:
    if t is None:
        return ctypes.c_void_p(0)
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError("tensors passed to the library must be contiguous device tensors")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def workspace_bytes(batch: Batch, budget: int, cand_mult: int = 4,
                    keep_tail: Optional[int] = None) -> int:
    tail = batch.w if keep_tail is None else keep_tail
    return int(lib().kv_workspace_bytes(batch.ref(), budget, cand_mult, tail))


def candidate_stride(batch: Batch, budget: int, cand_mult: int = 4,
                     keep_tail: Optional[int] = None) -> int:
    tail = batch.w if keep_tail is None else keep_tail
    return int(lib().kv_candidate_stride(batch.ref(), budget, cand_mult, tail))


def window_scores(batch: Batch, q_win, k, scale: float, row_max, row_sum, ws,
                  stream=None) -> None:
    _check(lib().kv_window_scores(batch.ref(), _ptr(q_win), _ptr(k), float(scale), _ptr(row_max),
                                  _ptr(row_sum), _ptr(ws), 0 if ws is None else ws.numel() *
                                  ws.element_size(), _stream(stream)), "kv_window_scores")


def mu_sigma(batch: Batch, q_win, k, scale: float, row_max, row_sum, mu, sigma, attn=None,
             stream=None) -> None:
    _check(lib().kv_mu_sigma(batch.ref(), _ptr(q_win), _ptr(k), float(scale), _ptr(row_max),
                             _ptr(row_sum), _ptr(mu), _ptr(sigma), _ptr(attn), _stream(stream)),
           "kv_mu_sigma")


def window_mu_sigma(batch: Batch, q_win, k, scale: float, row_max, row_sum, mu, sigma, ws,
                    stream=None) -> None:
    _check(lib().kv_window_mu_sigma(batch.ref(), _ptr(q_win), _ptr(k), float(scale),
                                    _ptr(row_max), _ptr(row_sum), _ptr(mu), _ptr(sigma), _ptr(ws),
                                    0 if ws is None else ws.numel() * ws.element_size(),
                                    _stream(stream)), "kv_window_mu_sigma")


def _sigma_rows(sigma_rows) -> int:
    return SIGMA_ROWS[sigma_rows] if isinstance(sigma_rows, str) else int(sigma_rows)


def mu_sigma_ex(batch: Batch, q_win, k, scale: float, row_max, row_sum, sigma_rows, mu, sigma,
                attn=None, stream=None) -> None:
    """kv_mu_sigma_ex; sigma_rows is "group_mean", "all_rows" or a KV_SIGMA_* value."""
    _check(lib().kv_mu_sigma_ex(batch.ref(), _ptr(q_win), _ptr(k), float(scale), _ptr(row_max),
                                _ptr(row_sum), _sigma_rows(sigma_rows), _ptr(mu), _ptr(sigma),
                                _ptr(attn), _stream(stream)), "kv_mu_sigma_ex")


def window_mu_sigma_ex(batch: Batch, q_win, k, scale: float, sigma_rows, row_max, row_sum, mu,
                       sigma, ws, stream=None) -> None:
    """kv_window_mu_sigma_ex; sigma_rows is "group_mean", "all_rows" or a KV_SIGMA_* value."""
    _check(lib().kv_window_mu_sigma_ex(batch.ref(), _ptr(q_win), _ptr(k), float(scale),
                                       _sigma_rows(sigma_rows), _ptr(row_max), _ptr(row_sum),
                                       _ptr(mu), _ptr(sigma), _ptr(ws),
                                       0 if ws is None else ws.numel() * ws.element_size(),
                                       _stream(stream)), "kv_window_mu_sigma_ex")


def window_mu_sigma_noalloc(batch: Batch, q_win, k, scale: float, row_max, row_sum, mu, sigma,
                            sigma_rows="group_mean", stream=None) -> None:
    """kv_window_mu_sigma_noalloc (no workspace: the library's static scratch)."""
    _check(lib().kv_window_mu_sigma_noalloc(batch.ref(), _ptr(q_win), _ptr(k), float(scale),
                                            _sigma_rows(sigma_rows), _ptr(row_max),
                                            _ptr(row_sum), _ptr(mu), _ptr(sigma),
                                            _stream(stream)), "kv_window_mu_sigma_noalloc")


def base_scores_workspace_bytes(batch: Batch) -> int:
    return int(lib().kv_base_scores_workspace_bytes(batch.ref()))


def window_base_scores(batch: Batch, q_win, k, scale: float, lambda1, row_max, row_sum, score,
                       w_mu: float = 1.0, sigma_rows="group_mean", ws=None, stream=None) -> None:
    """kv_window_base_scores."""
    _check(lib().kv_window_base_scores(batch.ref(), _ptr(q_win), _ptr(k), float(scale),
                                       _ptr(lambda1), float(w_mu), _sigma_rows(sigma_rows),
                                       _ptr(row_max), _ptr(row_sum), _ptr(score), _ptr(ws),
                                       0 if ws is None else ws.numel() * ws.element_size(),
                                       _stream(stream)), "kv_window_base_scores")


def _select_opts(pool, w_mu, budgets):
    if pool is None and w_mu is None and budgets is None:
        return None
    bh, bd = budgets.pointers() if budgets is not None else (None, None)
    return ctypes.byref(KvSelectOpts(1 if pool is None else int(pool),
                                     1.0 if w_mu is None else float(w_mu), bh, bd))


def mmr_select_scored(batch: Batch, score, k, v, lambda2, budget: int, cand_mult: int,
                      keep_tail: int, sel_idx, sel_score=None, cand_idx=None, cand_corr=None,
                      k_out=None, v_out=None, pool: Optional[int] = None,
                      budgets: Optional[Budgets] = None, stream=None) -> None:
    """kv_mmr_select_scored; with k_out / v_out the compaction runs in the same launch."""
    _check(lib().kv_mmr_select_scored(batch.ref(), _ptr(score), _ptr(k), _ptr(v), _ptr(lambda2),
                                      int(budget), int(cand_mult),
                                      int(keep_tail), _select_opts(pool, None, budgets),
                                      _ptr(sel_idx), _ptr(sel_score), _ptr(cand_idx),
                                      _ptr(cand_corr), _ptr(k_out), _ptr(v_out),
                                      _stream(stream)), "kv_mmr_select_scored")


def candidates_workspace_bytes(batch: Batch, budget: int, cand_mult: int, keep_tail: int,
                               w_mu: Optional[float] = None,
                               budgets: Optional[Budgets] = None) -> int:
    return int(lib().kv_candidates_workspace_bytes(batch.ref(), int(budget), int(cand_mult),
                                                   int(keep_tail),
                                                   _select_opts(None, w_mu, budgets)))


def window_candidates(batch: Batch, q_win, k, scale: float, lambda1, budget: int, cand_mult: int,
                      keep_tail: int, row_max, row_sum, ws, w_mu: Optional[float] = None,
                      budgets: Optional[Budgets] = None, sigma_rows="group_mean",
                      stream=None) -> None:
    """kv_window_candidates: row statistics out, the candidates into ws (see
    candidates_workspace_bytes) for mmr_select_candidates with the same selection arguments."""
    _check(lib().kv_window_candidates(batch.ref(), _ptr(q_win), _ptr(k), float(scale),
                                      _ptr(lambda1), _sigma_rows(sigma_rows), int(budget),
                                      int(cand_mult), int(keep_tail),
                                      _select_opts(None, w_mu, budgets), _ptr(row_max),
                                      _ptr(row_sum), _ptr(ws),
                                      0 if ws is None else ws.numel() * ws.element_size(),
                                      _stream(stream)), "kv_window_candidates")


def mmr_select_candidates(batch: Batch, ws, k, v, lambda2, budget: int, cand_mult: int,
                          keep_tail: int, sel_idx, sel_score=None, cand_idx=None, cand_corr=None,
                          k_out=None, v_out=None, w_mu: Optional[float] = None,
                          budgets: Optional[Budgets] = None, stream=None) -> None:
    """kv_mmr_select_candidates; with k_out / v_out the compaction runs in the same launch."""
    _check(lib().kv_mmr_select_candidates(batch.ref(), _ptr(ws),
                                          0 if ws is None else ws.numel() * ws.element_size(),
                                          _ptr(k), _ptr(v), _ptr(lambda2), int(budget),
                                          int(cand_mult), int(keep_tail),
                                          _select_opts(None, w_mu, budgets), _ptr(sel_idx),
                                          _ptr(sel_score), _ptr(cand_idx), _ptr(cand_corr),
                                          _ptr(k_out), _ptr(v_out), _stream(stream)),
           "kv_mmr_select_candidates")


def evict_pass(batch: Batch, q_win, k, v, scale: float, lambda1, lambda2, budget: int,
               cand_mult: int, keep_tail: int, row_max, row_sum, sel_idx, ws, sel_score=None,
               k_out=None, v_out=None, w_mu: Optional[float] = None,
               budgets: Optional[Budgets] = None, sigma_rows="group_mean", stream=None) -> None:
    """kv_evict_pass: window_candidates then mmr_select_candidates (with k_out / v_out the
    compaction), in one launch where the window kernel cuts the candidates and C <= 256."""
    _check(lib().kv_evict_pass(batch.ref(), _ptr(q_win), _ptr(k), _ptr(v), float(scale),
                               _ptr(lambda1), _ptr(lambda2), _sigma_rows(sigma_rows), int(budget),
                               int(cand_mult), int(keep_tail), _select_opts(None, w_mu, budgets),
                               _ptr(row_max), _ptr(row_sum), _ptr(sel_idx), _ptr(sel_score),
                               _ptr(k_out), _ptr(v_out), _ptr(ws),
                               0 if ws is None else ws.numel() * ws.element_size(),
                               _stream(stream)), "kv_evict_pass")


def mmr_select(batch: Batch, mu, sigma, k, lambda1, lambda2, budget: int, cand_mult: int,
               keep_tail: int, sel_idx, sel_score=None, cand_idx=None, cand_corr=None, ws=None,
               stream=None) -> None:
    _check(lib().kv_mmr_select(batch.ref(), _ptr(mu), _ptr(sigma), _ptr(k), _ptr(lambda1),
                               _ptr(lambda2), int(budget), int(cand_mult), int(keep_tail),
                               _ptr(sel_idx), _ptr(sel_score), _ptr(cand_idx), _ptr(cand_corr),
                               _ptr(ws), 0 if ws is None else ws.numel() * ws.element_size(),
                               _stream(stream)), "kv_mmr_select")


def mmr_select_compact(batch: Batch, mu, sigma, k, v, lambda1, lambda2, budget: int,
                       cand_mult: int, keep_tail: int, sel_idx, k_out, v_out, ws=None,
                       stream=None) -> None:
    _check(lib().kv_mmr_select_compact(batch.ref(), _ptr(mu), _ptr(sigma), _ptr(k), _ptr(v),
                                       _ptr(lambda1), _ptr(lambda2), int(budget), int(cand_mult),
                                       int(keep_tail), _ptr(sel_idx), _ptr(k_out), _ptr(v_out),
                                       _ptr(ws), 0 if ws is None else ws.numel() * ws.element_size(),
                                       _stream(stream)), "kv_mmr_select_compact")


def mmr_select_ex(batch: Batch, mu, sigma, k, lambda1, lambda2, budget: int, cand_mult: int,
                  keep_tail: int, sel_idx, sel_score=None, cand_idx=None, cand_corr=None, ws=None,
                  pool: Optional[int] = None, w_mu: Optional[float] = None,
                  budgets: Optional[Budgets] = None, stream=None) -> None:
    """kv_mmr_select_ex; options are passed as NULL when pool, w_mu and budgets are all None.
    With `budgets`, `budget` is the row stride of sel_idx / sel_score."""
    opts = _select_opts(pool, w_mu, budgets)
    _check(lib().kv_mmr_select_ex(batch.ref(), _ptr(mu), _ptr(sigma), _ptr(k), _ptr(lambda1),
                                  _ptr(lambda2), int(budget), int(cand_mult), int(keep_tail), opts,
                                  _ptr(sel_idx), _ptr(sel_score), _ptr(cand_idx),
                                  _ptr(cand_corr), _ptr(ws),
                                  0 if ws is None else ws.numel() * ws.element_size(),
                                  _stream(stream)), "kv_mmr_select_ex")


def compact_cache(batch: Batch, k, v, sel_idx, budget: int, keep_tail: int, k_out, v_out,
                  stream=None) -> None:
    _check(lib().kv_compact_cache(batch.ref(), _ptr(k), _ptr(v), _ptr(sel_idx), int(budget),
                                  int(keep_tail), _ptr(k_out), _ptr(v_out), _stream(stream)),
           "kv_compact_cache")


def compact_cache_ex(batch: Batch, k, v, sel_idx, budget: int, keep_tail: int,
                     budgets: Optional[Budgets], k_out, v_out, out_rows: int = 0,
                     stream=None) -> None:
    bh, bd = budgets.pointers() if budgets is not None else (None, None)
    _check(lib().kv_compact_cache_ex(batch.ref(), _ptr(k), _ptr(v), _ptr(sel_idx), int(budget),
                                     int(keep_tail), bh, bd, int(out_rows), _ptr(k_out),
                                     _ptr(v_out), _stream(stream)), "kv_compact_cache_ex")


class CacheBatch:
    """Shape of a batch of caches for decoding (kv_cache_batch): per-problem lengths on the host
    and the device.  `advance()` adds one row to every length (after a call that appended)."""

    def __init__(self, dtype: str, h_q: int, h_kv: int, d: int, row_stride: int,
                 lens: Sequence[int], device=None):
        import torch
        self.dtype_name = dtype
        self.h_q, self.h_kv, self.d, self.row_stride = int(h_q), int(h_kv), int(d), int(row_stride)
        self.lens_host = np.ascontiguousarray(np.asarray(lens, dtype=np.int32))
        self._dev = torch.device("cuda") if device is None else torch.device(device)
        self._sync()

    def _sync(self):
        import torch
        self.lens_dev = torch.from_numpy(self.lens_host).to(self._dev)
        self.struct = KvCacheBatch(KV_BF16 if self.dtype_name == "bf16" else KV_F32,
                                   len(self.lens_host), self.h_q, self.h_kv, self.d,
                                   self.row_stride, self.lens_host.ctypes.data,
                                   self.lens_dev.data_ptr())

    def advance(self):
        self.lens_host = self.lens_host + 1
        self._sync()

    @property
    def n_prob(self) -> int:
        return len(self.lens_host)

    def ref(self):
        return ctypes.byref(self.struct)


def decode_workspace_bytes(cb: CacheBatch) -> int:
    return int(lib().kv_decode_workspace_bytes(cb.ref()))


def decode_attention(cb: CacheBatch, q, k_cache, v_cache, k_new, v_new, scale: float, out,
                     ws=None, stream=None) -> None:
    _check(lib().kv_decode_attention(cb.ref(), _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(k_new),
                                     _ptr(v_new), float(scale), _ptr(out), _ptr(ws),
                                     0 if ws is None else ws.numel() * ws.element_size(),
                                     _stream(stream)), "kv_decode_attention")


def pyramid_budgets(budget: int, n_layers: int, beta: float) -> np.ndarray:
    """Depth-decreasing per-layer budgets at the total of a uniform `budget` (int32)."""
    out = (ctypes.c_int32 * n_layers)()
    _check(lib().kv_pyramid_budgets(int(budget), int(n_layers), float(beta), out),
           "kv_pyramid_budgets")
    return np.frombuffer(out, dtype=np.int32).copy()


def depth_profile(family: str, params: Sequence[float], n_layers: int) -> np.ndarray:
    """lambda per layer (float32) from a Global / Segments / Curve latent profile."""
    fam = PROFILE_FAMILIES[family] if isinstance(family, str) else int(family)
    p = (ctypes.c_double * len(params))(*[float(x) for x in params])
    out = (ctypes.c_float * n_layers)()
    _check(lib().kv_depth_profile(fam, p, len(params), int(n_layers), out), "kv_depth_profile")
    return np.frombuffer(out, dtype=np.float32).copy()
