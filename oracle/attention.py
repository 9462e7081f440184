"""Chunk prefill attention over the compacted history plus the chunk itself (oracle, float64).

Paper passages followed:
  * Background, omni model architecture: during prefill the backbone computes the new input's
    KV states, appends them to the cache and attends over the cached history.
  * Fragmentation after logical eviction / retention-aware paging: attention runs over the KV
    slots presented to it; after eager packing these are the contiguous rows [0, n_ctx).

Readings where the paper is silent:
  * Causal mask anchored bottom-right: chunk query i (0 <= i < L) sees keys j <= n_ctx - L + i.
  * Grouped-query attention with contiguous groups: query head h reads KV head h // (H_q/H_kv).
  * Scale 1/sqrt(d); no rotary embedding, soft-capping or dropout inside the operation.
"""
from __future__ import annotations

import numpy as np

from .omnipick import to_f64  # noqa: F401  (re-exported)


def chunk_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float) -> np.ndarray:
    """softmax(scale * q k^T + causal mask) v in float64.

    q: [L, H_q, d]; k, v: [n_ctx, H_kv, d] (rows [0, n_ctx) of the compacted pool, chunk last).
    Returns [L, H_q, d] float64.
    """
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    L, Hq, d = q.shape
    n_ctx, Hkv, _ = k.shape
    group = Hq // Hkv
    kept = n_ctx - L
    if kept < 0:
        raise ValueError("pool shorter than the chunk")
    visible = np.arange(n_ctx)[None, :] <= (kept + np.arange(L))[:, None]   # [L, n_ctx]
    out = np.empty((L, Hq, d), np.float64)
    for h in range(Hq):
        g = h // group
        s = scale * (q[:, h, :] @ k[:, g, :].T)
        s = np.where(visible, s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=1, keepdims=True)
        out[:, h, :] = p @ v[:, g, :]
    return out
