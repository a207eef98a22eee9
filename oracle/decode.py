"""Attention of a newly generated token over the compacted cache (section 4.3: after eviction the
model generates tokens against the B + W kept rows of every layer, and the paper times prefill
plus generation end to end).

TEST INFRASTRUCTURE ONLY (see the package docstring).

This is ordinary scaled dot-product attention for one query token per head, written out in
float64 from the exact values of the stored inputs.  Query head h reads kv head h // G
(G = h_q / h_kv).  If the new token's own key and value are given they are appended to the cache
first, so the token also attends to itself.
"""
from __future__ import annotations

from typing import Optional

import numpy as np


def decode_attention(q: np.ndarray, k_rows: np.ndarray, v_rows: np.ndarray, scale: float,
                     k_new: Optional[np.ndarray] = None,
                     v_new: Optional[np.ndarray] = None) -> np.ndarray:
    """q [h_q, d]; k_rows, v_rows [h_kv, n, d] (the cache rows in use); k_new, v_new [h_kv, d] or
    None.  Returns o [h_q, d] = softmax(scale q K^T) V per query head, in float64."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k_rows, dtype=np.float64)
    v = np.asarray(v_rows, dtype=np.float64)
    if k_new is not None:
        k = np.concatenate([k, np.asarray(k_new, dtype=np.float64)[:, None, :]], axis=1)
        v = np.concatenate([v, np.asarray(v_new, dtype=np.float64)[:, None, :]], axis=1)
    h_q = q.shape[0]
    h_kv = k.shape[0]
    group = h_q // h_kv
    out = np.empty((h_q, q.shape[1]))
    for h in range(h_q):
        g = h // group
        logits = scale * (k[g] @ q[h])
        w = np.exp(logits - logits.max())
        out[h] = (w / w.sum()) @ v[g]
    return out
