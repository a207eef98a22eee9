"""Seeded synthetic inputs for the post-prefill eviction-scoring path.

This module only draws inputs: window queries, cached keys and values, context lengths and the
per-layer coefficient profile *specifications* (family and latent parameters).  It computes none of
the method's arithmetic (no attention, statistics, scores, selection or profile evaluation), so both
the HIP path and the CPU oracle can take their inputs from here.

Shapes follow the workloads the paper evaluates (Mistral-7B: 32 layers, 32 query heads sharing 8
key/value heads, head dimension 128; prompts of several thousand to ~32k tokens, section 4.1 and
the efficiency discussion in section 4.3).  The value structure stands in for the phenomena that
motivate the score (section 1): an attention sink, clusters of near-duplicate salient keys, and for
the retrieval-style layout, passages that occur twice in the prompt.

Recipe (per problem = one (sequence, layer), seed ``[config_id, sequence, layer]``):
  * window queries q[h, r, :] ~ N(0, 1) / sqrt(d);
  * bulk keys ~ N(0, 1) / sqrt(d);
  * per kv-head g, the salience direction u_g is the normalised sum of the group's window queries and
    nu_g the mean of q . u_g over those queries.  A key c * (u_g + 2 xi) with xi a random unit vector
    orthogonal to u_g has a mean window logit of c * scale * nu_g, so c(alpha) = alpha / (scale * nu_g)
    plants a mean logit of alpha nats while xi spreads the logit across window queries;
  * sink at position 0: c(6) * u_g;
  * each near-duplicate cluster is a contiguous region whose members are one base key plus independent
    N(0, (0.05 * rms(base))^2) noise per entry (5 % relative noise, cosine ~0.9988 to the base);
  * a passage is a region of distinct salient keys; its second occurrence copies it with the same 5 %
    noise;
  * regions are placed at random, non-overlapping offsets in [1, L - W);
  * values are random bf16 numbers (random sign and mantissa, exponent 2^-7..2^2): they are only ever
    gathered, never used in arithmetic;
  * optionally, given positions of given kv heads are re-drawn after planting: their keys are
    replaced by fresh bulk keys N(0, 1) / sqrt(d) from the seed
    ``[config_id, sequence, layer, 1000 + kv_head, position, n]`` (n counts earlier re-draws of the
    same position).  The positions come from the caller; this module only draws.

Decode over compacted caches (draw_decode): queries, keys, values and the new token's key/value
~ N(0, 1), a few rows of every block's keys scaled by 4 (dominant rows), scale 1/sqrt(d).

bf16 tensors are returned as their raw uint16 bit patterns (round-to-nearest-even from fp32).
"""
from __future__ import annotations

import concurrent.futures
import dataclasses
import os
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

F32 = "f32"
BF16 = "bf16"

PROFILE_GLOBAL = "global"
PROFILE_SEGMENTS = "segments"
PROFILE_CURVE = "curve"

NOISE_REL = 0.05
SINK_ALPHA = 6.0


@dataclasses.dataclass(frozen=True)
class ProfileSpec:
    """A depth-profile family and its latent parameters a (lambda = sinh(a(layer)))."""
    family: str
    params: Tuple[float, ...]


@dataclasses.dataclass(frozen=True)
class Layout:
    """Planted structure of one problem's keys."""
    n_clusters: int = 0
    cluster_size: int = 16
    cluster_alpha: Tuple[float, float] = (2.0, 4.0)
    n_passages: int = 0
    passage_len: int = 128
    passage_alpha: Tuple[float, float] = (0.5, 2.0)
    cluster_density: Optional[float] = None  # if set, n_clusters = floor(density * L / size)
    noise_rel: float = NOISE_REL  # relative noise of cluster members and passage copies (0: exact)


@dataclasses.dataclass
class Workload:
    name: str
    config_id: int
    dtype: str
    h_q: int
    h_kv: int
    d: int
    w: int
    budget: int
    n_seq: int
    n_layers: int
    seq_lens: List[int]
    layout: Layout
    lam1: ProfileSpec
    lam2: ProfileSpec

    @property
    def n_prob(self) -> int:
        return self.n_seq * self.n_layers

    @property
    def lens(self) -> np.ndarray:
        """Context length of every problem p = sequence * n_layers + layer."""
        return np.repeat(np.asarray(self.seq_lens, dtype=np.int32), self.n_layers)

    @property
    def tok_off(self) -> np.ndarray:
        """Packed token offset of every problem (exclusive prefix sum of the lengths)."""
        lens = self.lens.astype(np.int64)
        off = np.zeros_like(lens)
        off[1:] = np.cumsum(lens)[:-1]
        return off

    @property
    def scale(self) -> float:
        return float(1.0 / np.sqrt(self.d))

    def layer_of(self, p: int) -> int:
        return p % self.n_layers

    def seq_of(self, p: int) -> int:
        return p // self.n_layers


# --------------------------------------------------------------------------------------------
# Named workloads (Mistral-7B attention layout unless stated)
# --------------------------------------------------------------------------------------------

def _a(x: float) -> float:
    # Latent parameter of a stated coefficient: lambda = sinh(a)  <=>  a = asinh(lambda).
    return float(np.arcsinh(x))


def tiny_f32() -> Workload:
    """fp32, one layer, 2 query heads sharing 1 kv head, d=64, L=512, W=8, B=16."""
    return Workload("tiny_f32_L512_W8_B16", 0, F32, 2, 1, 64, 8, 16, 1, 1, [512],
                    Layout(n_clusters=4, cluster_size=8),
                    ProfileSpec(PROFILE_GLOBAL, (_a(0.5),)), ProfileSpec(PROFILE_GLOBAL, (_a(-1.0),)))


def mistral_layer() -> Workload:
    """bf16, one Mistral-7B-shaped layer, L=4096, W=32, B=64, 16 clusters of 16."""
    return Workload("mistral_layer_L4096_W32_B64", 1, BF16, 32, 8, 128, 32, 64, 1, 1, [4096],
                    Layout(n_clusters=16, cluster_size=16),
                    ProfileSpec(PROFILE_GLOBAL, (_a(0.3),)), ProfileSpec(PROFILE_GLOBAL, (_a(-0.8),)))


def mistral_pass_8k(budget: int = 64, n_layers: int = 32, L: int = 8192) -> Workload:
    """bf16, 32 layers, L=8192, W=32, three-segment lambda2 = -1.0/-0.5/-1.2, lambda1 = 0.2."""
    return Workload(f"mistral32_L{L}_W32_B{budget}" if n_layers == 32 else
                    f"mistral{n_layers}_L{L}_W32_B{budget}", 2, BF16, 32, 8, 128, 32, budget, 1,
                    n_layers, [L], Layout(cluster_density=0.02, cluster_size=16),
                    ProfileSpec(PROFILE_GLOBAL, (_a(0.2),)),
                    ProfileSpec(PROFILE_SEGMENTS, (_a(-1.0), _a(-0.5), _a(-1.2))))


# Quadratic latent profile for lambda2 with a mid-layer sign flip: a(t) = c0 + c1 t + c2 t^2 is
# positive for t in (0.371, 0.661), i.e. layers 12..20 of 32 (peak lambda2 ~ +0.127 at layer 16).
CURVE_32K = (-1.47190, 6.19355, -6.0)


def mistral_pass_32k(n_layers: int = 32, L: int = 32768, n_clusters: int = 64,
                     n_passages: int = 30) -> Workload:
    """bf16, 32 layers, L=32768, W=32, B=64, quadratic lambda2 profile, lambda1 = 0.2."""
    name = (f"mistral32_L{L}_W32_B64" if (n_layers == 32 and L == 32768)
            else f"mistral{n_layers}_L{L}_W32_B64")
    return Workload(name, 3, BF16, 32, 8, 128, 32, 64, 1, n_layers, [L],
                    Layout(n_clusters=n_clusters, cluster_size=16, n_passages=n_passages,
                           passage_len=128),
                    ProfileSpec(PROFILE_GLOBAL, (_a(0.2),)), ProfileSpec(PROFILE_CURVE, CURVE_32K))


RAGGED_RUNS = {  # (lambda1, lambda2) of the three term-ablation runs
    "dispersion_only": (0.3, 0.0),
    "redundancy_only": (0.0, -0.15),
    "both": (0.3, -0.15),
}


def ragged_batch(run: str = "both", n_seq: int = 8, n_layers: int = 32,
                 len_range: Tuple[int, int] = (2048, 31744)) -> Workload:
    """bf16 ragged batch of n_seq sequences with L ~ U{2048..31744}, 32 layers, W=32, B=128."""
    lam1, lam2 = RAGGED_RUNS[run]
    lens = np.random.default_rng([4, 0]).integers(len_range[0], len_range[1] + 1, n_seq)
    name = f"ragged{n_seq}x{n_layers}_L{len_range[0]}-{len_range[1]}_W32_B128_{run}"
    return Workload(name, 4, BF16, 32, 8, 128, 32, 128, n_seq, n_layers,
                    [int(x) for x in lens], Layout(cluster_density=0.02, cluster_size=16),
                    ProfileSpec(PROFILE_GLOBAL, (_a(lam1),)), ProfileSpec(PROFILE_GLOBAL, (_a(lam2),)))


# --------------------------------------------------------------------------------------------
# Drawing
# --------------------------------------------------------------------------------------------

def f32_to_bf16_bits(x: np.ndarray, out: Optional[np.ndarray] = None,
                     inplace: bool = False) -> np.ndarray:
    """Round fp32 to bf16 (nearest, ties to even) and return the uint16 bit patterns.

    With inplace=True the float32 input is used as scratch (its contents are destroyed)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    b = x.view(np.uint32) if inplace else x.view(np.uint32).copy()
    r = b >> np.uint32(16)
    r &= np.uint32(1)
    r += np.uint32(0x7FFF)
    b += r
    b >>= np.uint32(16)
    if out is None:
        return b.astype(np.uint16)
    np.copyto(out, b.reshape(out.shape), casting="unsafe")
    return out


def _unit_orthogonal(rng: np.random.Generator, u: np.ndarray, n: int) -> np.ndarray:
    x = rng.standard_normal((n, u.shape[0]))
    x -= np.outer(x @ u, u)
    x /= np.linalg.norm(x, axis=1, keepdims=True)
    return x


def _place(rng: np.random.Generator, lo: int, hi: int, lengths: Sequence[int]) -> List[int]:
    """Random non-overlapping starts of regions with the given lengths inside [lo, hi)."""
    total = int(sum(lengths))
    free = (hi - lo) - total
    if free < 0:
        raise ValueError("planted regions do not fit into the context")
    order = rng.permutation(len(lengths))
    gaps = rng.multinomial(free, np.full(len(lengths) + 1, 1.0 / (len(lengths) + 1)))
    starts = [0] * len(lengths)
    pos = lo
    for slot, idx in enumerate(order):
        pos += int(gaps[slot])
        starts[idx] = pos
        pos += int(lengths[idx])
    return starts


def _planted_keys(rng, q_group: np.ndarray, scale: float, L: int, w: int, lay: Layout,
                  n_clusters: int, k: np.ndarray) -> None:
    """Overwrite rows of one kv-head's keys k[L, d] (float32) with the planted structure (computed
    in float64, stored rounded)."""
    d = k.shape[1]
    u = q_group.sum(axis=0)
    u /= np.linalg.norm(u)
    nu = float((q_group @ u).mean())
    c = lambda alpha: alpha / (scale * nu)  # noqa: E731
    k[0] = c(SINK_ALPHA) * u
    lengths: List[int] = [lay.cluster_size] * n_clusters
    lengths += [lay.passage_len] * (2 * lay.n_passages)
    if not lengths:
        return
    starts = _place(rng, 1, L - w, lengths)
    if n_clusters:
        alphas = np.linspace(lay.cluster_alpha[0], lay.cluster_alpha[1], n_clusters)
        xi = _unit_orthogonal(rng, u, n_clusters)
        for ci in range(n_clusters):
            base = c(alphas[ci]) * (u + 2.0 * xi[ci])
            rms = np.linalg.norm(base) / np.sqrt(d)
            m = lay.cluster_size
            k[starts[ci]:starts[ci] + m] = base + lay.noise_rel * rms * rng.standard_normal((m, d))
    if lay.n_passages:
        alphas = np.linspace(lay.passage_alpha[0], lay.passage_alpha[1], lay.n_passages)
        for pi in range(lay.n_passages):
            n = lay.passage_len
            xi = _unit_orthogonal(rng, u, n)
            toks = c(alphas[pi]) * (u[None, :] + 2.0 * xi)
            rms = np.linalg.norm(toks, axis=1, keepdims=True) / np.sqrt(d)
            s0 = starts[n_clusters + 2 * pi]
            s1 = starts[n_clusters + 2 * pi + 1]
            k[s0:s0 + n] = toks
            k[s1:s1 + n] = toks + lay.noise_rel * rms * rng.standard_normal((n, d))


def _random_values(rng: np.random.Generator, shape, out: Optional[np.ndarray] = None) -> np.ndarray:
    """Random bf16 bit patterns: random sign and mantissa, exponent in [2^-7, 2^2]."""
    n = int(np.prod(shape))
    raw = np.frombuffer(rng.bytes(2 * n), dtype=np.uint16).copy()
    expo = raw >> np.uint16(7)
    expo %= np.uint16(10)
    expo += np.uint16(120)
    expo <<= np.uint16(7)
    raw &= np.uint16(0x807F)  # sign and mantissa
    raw |= expo
    if out is None:
        return raw.reshape(shape)
    np.copyto(out, raw.reshape(out.shape))
    return out


@dataclasses.dataclass
class ProblemInputs:
    """Inputs of one problem, stored as they are handed to the kernels (f32 or bf16 bits)."""
    q_win: np.ndarray  # [h_q, w, d]
    k: np.ndarray      # [h_kv, L, d]
    v: np.ndarray      # [h_kv, L, d]


def draw_problem(wl: Workload, p: int, k_out: Optional[np.ndarray] = None,
                 v_out: Optional[np.ndarray] = None,
                 redraw: Optional[Dict[int, Sequence[int]]] = None) -> ProblemInputs:
    """Draw the inputs of problem p (deterministic in (config_id, sequence, layer)).

    k_out / v_out (optional, [h_kv, L, d] in the stored dtype) receive K and V directly.  redraw
    (optional): {kv_head: [position, ...]} keys to replace by fresh bulk keys after planting, in
    list order (a position listed twice is re-drawn twice)."""
    s, layer = wl.seq_of(p), wl.layer_of(p)
    L = int(wl.seq_lens[s])
    rng = np.random.default_rng([wl.config_id, s, layer])
    d, w, h_q, h_kv = wl.d, wl.w, wl.h_q, wl.h_kv
    g_sz = h_q // h_kv
    q = rng.standard_normal((h_q, w, d), dtype=np.float32)
    q /= np.float32(np.sqrt(d))
    k = rng.standard_normal((h_kv, L, d), dtype=np.float32)
    k /= np.float32(np.sqrt(d))
    lay = wl.layout
    n_clusters = lay.n_clusters
    if lay.cluster_density is not None:
        n_clusters = int(np.floor(lay.cluster_density * L / lay.cluster_size))
    for g in range(h_kv):
        qg = q[g * g_sz:(g + 1) * g_sz].reshape(-1, d).astype(np.float64)
        _planted_keys(rng, qg, wl.scale, L, w, lay, n_clusters, k[g])
    for g, positions in (redraw or {}).items():
        count: Dict[int, int] = {}
        for pos in positions:
            pos = int(pos)
            if not 0 <= pos < L:
                raise ValueError(f"re-drawn position {pos} outside [0, {L})")
            n = count.get(pos, 0)
            count[pos] = n + 1
            r2 = np.random.default_rng([wl.config_id, s, layer, 1000 + int(g), pos, n])
            k[int(g), pos] = r2.standard_normal(d, dtype=np.float32) / np.float32(np.sqrt(d))
    if wl.dtype == F32:
        v = rng.standard_normal((h_kv, L, d), dtype=np.float32)
        if k_out is not None:
            np.copyto(k_out, k)
            k = k_out
        if v_out is not None:
            np.copyto(v_out, v)
            v = v_out
        return ProblemInputs(q, k, v)
    v = _random_values(rng, (h_kv, L, d), v_out)
    kb = f32_to_bf16_bits(k, k_out, inplace=True)
    return ProblemInputs(f32_to_bf16_bits(q), kb, v)


@dataclasses.dataclass
class PackedInputs:
    """All problems of a workload packed the way the C ABI expects them."""
    q_win: np.ndarray   # [n_prob, h_q, w, d]
    k: np.ndarray       # flat, problem p at tok_off[p]*h_kv*d, layout [h_kv][L_p][d]
    v: np.ndarray
    lens: np.ndarray    # int32 [n_prob]
    tok_off: np.ndarray  # int64 [n_prob]


def draw_packed(wl: Workload, problems: Optional[Sequence[int]] = None,
                threads: Optional[int] = None,
                redraw: Optional[Dict[int, Dict[int, Sequence[int]]]] = None) -> PackedInputs:
    """Draw and pack the given problems (default: all) of a workload (problems are independent
    and drawn in parallel threads; the result does not depend on the thread count).  redraw:
    {problem: {kv_head: [position, ...]}}, see draw_problem."""
    probs = list(range(wl.n_prob)) if problems is None else list(problems)
    lens = np.asarray([wl.seq_lens[wl.seq_of(p)] for p in probs], dtype=np.int32)
    off = np.zeros(len(probs), dtype=np.int64)
    if len(probs) > 1:
        off[1:] = np.cumsum(lens.astype(np.int64))[:-1]
    elt = np.float32 if wl.dtype == F32 else np.uint16
    total = int(lens.astype(np.int64).sum()) * wl.h_kv * wl.d
    k = np.empty(total, dtype=elt)
    v = np.empty(total, dtype=elt)
    q = np.empty((len(probs), wl.h_q, wl.w, wl.d), dtype=elt)

    def one(j: int) -> None:
        n = int(lens[j]) * wl.h_kv * wl.d
        base = int(off[j]) * wl.h_kv * wl.d
        shape = (wl.h_kv, int(lens[j]), wl.d)
        pi = draw_problem(wl, probs[j], k[base:base + n].reshape(shape),
                          v[base:base + n].reshape(shape), (redraw or {}).get(probs[j]))
        q[j] = pi.q_win

    workers = max(1, min(len(probs), threads if threads else min(16, os.cpu_count() or 1)))
    if workers == 1:
        for j in range(len(probs)):
            one(j)
    else:
        with concurrent.futures.ThreadPoolExecutor(workers) as ex:
            list(ex.map(one, range(len(probs))))
    return PackedInputs(q, k, v, lens, off)


def all_workloads() -> List[Workload]:
    return [tiny_f32(), mistral_layer(), mistral_pass_8k(32), mistral_pass_8k(64),
            mistral_pass_8k(128), mistral_pass_32k(), ragged_batch("dispersion_only"),
            ragged_batch("redundancy_only"), ragged_batch("both")]


# --------------------------------------------------------------------------------------------
# Decode over compacted caches
# --------------------------------------------------------------------------------------------

@dataclasses.dataclass
class DecodeInputs:
    """A batch of caches in the block layout of kv_cache_batch plus one generated token each.

    q [n_prob, h_q, d]; k, v [n_prob, h_kv, row_stride, d] (every row filled, rows >= len too);
    k_new, v_new [n_prob, h_kv, d]; bf16 as uint16 bit patterns."""
    dtype: str
    h_q: int
    h_kv: int
    d: int
    row_stride: int
    lens: np.ndarray
    q: np.ndarray
    k: np.ndarray
    v: np.ndarray
    k_new: np.ndarray
    v_new: np.ndarray

    @property
    def scale(self) -> float:
        return float(1.0 / np.sqrt(self.d))


def draw_decode(dtype: str, h_q: int, h_kv: int, d: int, row_stride: int, lens: Sequence[int],
                seed: int = 0, peak_rows: int = 4) -> DecodeInputs:
    """Random queries, keys and values ~ N(0, 1); in every block `peak_rows` rows of K are scaled
    by 4 so that the softmax has a few dominant rows, as attention to kept heavy hitters does."""
    rng = np.random.default_rng([7, seed])
    n = len(lens)
    k = rng.standard_normal((n, h_kv, row_stride, d)).astype(np.float32)
    for p in range(n):
        for g in range(h_kv):
            rows = rng.integers(0, max(1, int(lens[p])), peak_rows)
            k[p, g, rows] *= 4.0
    v = rng.standard_normal((n, h_kv, row_stride, d)).astype(np.float32)
    q = rng.standard_normal((n, h_q, d)).astype(np.float32)
    k_new = rng.standard_normal((n, h_kv, d)).astype(np.float32)
    v_new = rng.standard_normal((n, h_kv, d)).astype(np.float32)
    if dtype == BF16:
        k, v, q, k_new, v_new = (f32_to_bf16_bits(x) for x in (k, v, q, k_new, v_new))
    return DecodeInputs(dtype, h_q, h_kv, d, row_stride, np.asarray(lens, dtype=np.int32), q, k,
                        v, k_new, v_new)
