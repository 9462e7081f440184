"""Pins for the oracle's chunk attention: brute force, torch SDPA in float64, closed-form special
cases, and the full-budget invariant (the whole step reproduces dense causal attention)."""
import math

import numpy as np
import pytest
import torch

import oracle
import streamgen as sg
from tests._util import storage_np


def _rand(seed, L, n_ctx, Hq, Hkv, d):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((L, Hq, d)), rng.standard_normal((n_ctx, Hkv, d)),
            rng.standard_normal((n_ctx, Hkv, d)))


def test_brute_force_triple_loop():
    q, k, v = _rand(0, 3, 5, 4, 2, 3)
    scale = 0.7
    out = oracle.chunk_attention(q, k, v, scale)
    L, n = 3, 5
    for i in range(L):
        for h in range(4):
            g = h // 2
            lim = n - L + i
            w = [math.exp(scale * sum(q[i, h, t] * k[j, g, t] for t in range(3)))
                 for j in range(lim + 1)]
            z = sum(w)
            for t in range(3):
                ref = sum(w[j] * v[j, g, t] for j in range(lim + 1)) / z
                assert abs(out[i, h, t] - ref) < 1e-12


@pytest.mark.parametrize("L,n,Hq,Hkv,d", [(7, 30, 8, 2, 16), (1, 1, 4, 1, 8), (16, 16, 6, 3, 4)])
def test_matches_torch_sdpa_float64(L, n, Hq, Hkv, d):
    q, k, v = _rand(1, L, n, Hq, Hkv, d)
    scale = 1.0 / math.sqrt(d)
    out = oracle.chunk_attention(q, k, v, scale)
    G = Hq // Hkv
    qt = torch.from_numpy(q).permute(1, 0, 2)                        # [Hq, L, d]
    kt = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(G, 0)
    vt = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(G, 0)
    mask = torch.arange(n)[None, :] <= (n - L + torch.arange(L))[:, None]
    ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask, scale=scale)
    assert np.abs(out - ref.permute(1, 0, 2).numpy()).max() < 1e-12


def test_rows_sum_to_one():
    q, k, _ = _rand(2, 9, 40, 4, 1, 8)
    out = oracle.chunk_attention(q, k, np.ones((40, 1, 8)), 0.5)
    assert np.abs(out - 1.0).max() < 1e-12


def test_single_query_no_history_returns_its_value():
    q, k, v = _rand(3, 1, 1, 4, 2, 8)
    out = oracle.chunk_attention(q, k, v, 0.3)
    assert np.array_equal(out[0], np.repeat(v[0], 2, axis=0))


def test_identical_keys_average_visible_values():
    q, k, v = _rand(4, 4, 10, 2, 1, 8)
    k[:] = k[0]
    out = oracle.chunk_attention(q, k, v, 0.3)
    for i in range(4):
        assert np.abs(out[i, 0] - v[: 6 + i + 1, 0].mean(0)).max() < 1e-12


def test_full_budget_step_is_dense_causal_attention():
    units = [(1, 20), (2, 7), (3, 9), (1, 20), (2, 7)]
    cfg, lay, seg = sg.custom_stream(units, [(1, 6), (2, 3)], n_q_heads=4, n_kv_heads=2,
                                     head_dim=16, budget=10 ** 4, recent=9)
    st = oracle.stream_step(storage_np(seg.k_hist), storage_np(seg.v_hist), "bf16", lay.unit_id,
                            lay.modality, lay.pos, lay.n_units, cfg.weights, cfg.budget,
                            cfg.recent, storage_np(seg.k_chunk), storage_np(seg.v_chunk),
                            lay.chunk_modality, lay.chunk_unit, storage_np(seg.q), cfg.scale,
                            10 ** 4, 64)
    assert st["keep"].all()
    kd = np.concatenate([oracle.to_f64(storage_np(seg.k_hist), "bf16"),
                         oracle.to_f64(storage_np(seg.k_chunk), "bf16")])
    vd = np.concatenate([oracle.to_f64(storage_np(seg.v_hist), "bf16"),
                         oracle.to_f64(storage_np(seg.v_chunk), "bf16")])
    dense = oracle.chunk_attention(oracle.to_f64(storage_np(seg.q), "bf16"), kd, vd, cfg.scale)
    assert np.array_equal(st["out"], dense)
