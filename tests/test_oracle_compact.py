"""Pins for the oracle's eager compaction: a hand-worked case, identity at full retention,
order preservation, verbatim rows, and the paper's printed physical-span figures."""
import json
import os

import numpy as np
import pytest

import oracle
from oracle import CapacityError
import streamgen as sg
from tests._util import storage_np


def test_hand_worked_example(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "compact_worked_example.json")))
    n = len(g["unit_id"])
    k = np.arange(n * 2 * 4, dtype=np.float32).reshape(n, 2, 4)
    kc = -np.arange(2 * 2 * 4, dtype=np.float32).reshape(2, 2, 4) - 1
    cp = oracle.compact_kv(k, k + 0.5, g["unit_id"], g["modality"], g["pos"], g["keep"],
                           g["n_units"], kc, kc - 0.5, g["chunk_modality"], g["chunk_unit"],
                           100, g["page_size"])
    assert cp["src_of_dst"].tolist() == g["expected_src_of_dst"]
    assert cp["unit_id"].tolist() == g["expected_unit_id"]
    assert cp["modality"].tolist() == g["expected_modality"]
    assert cp["pos"].tolist() == g["expected_pos"]
    assert cp["unit_remap"].tolist() == g["expected_unit_remap"]
    assert cp["n_ctx"] == g["expected_n_ctx"] and cp["n_pages"] == g["expected_n_pages"]
    assert np.array_equal(cp["k"][:6], k[[0, 1, 7, 9, 10, 11]])
    assert np.array_equal(cp["k"][6:], kc) and np.array_equal(cp["v"][6:], kc - 0.5)


def test_paper_span_figures(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "paper_spans.json")))
    for c in g["cuda_spans"]:
        assert oracle.page_span(c["useful"], c["page"]) == c["compacted_span"]
        assert c["native_span"] % c["page"] == 0 and c["native_span"] > c["compacted_span"]
        assert round(100 * (1 - c["compacted_span"] / c["native_span"]), 1) == c["reduction_pct"]
    m = g["metal_eager_vs_native"]
    assert oracle.page_span(m["eager_span"], m["page"]) == m["eager_span"]
    assert m["native_span"] / m["eager_span"] == m["ratio"]
    assert oracle.n_pages(0, 64) == 0 and oracle.n_pages(1, 64) == 1 and oracle.n_pages(64, 64) == 1
    assert oracle.n_pages(65, 64) == 2


def _case(seed, evict=0.0):
    rng = np.random.default_rng(seed)
    units = sg.random_units(rng, int(rng.integers(2, 30)))
    evicted = set(np.flatnonzero(rng.random(len(units)) < evict).tolist())
    cfg, lay, seg = sg.custom_stream(units, [(1, 5), (2, 3)], seed=seed, evicted=evicted)
    return cfg, lay, seg, rng


def test_keep_all_is_identity():
    cfg, lay, seg, _ = _case(5)
    k = storage_np(seg.k_hist)
    cp = oracle.compact_kv(k, storage_np(seg.v_hist), lay.unit_id, lay.modality, lay.pos,
                           np.ones(lay.n_units, np.uint8), lay.n_units, storage_np(seg.k_chunk),
                           storage_np(seg.v_chunk), lay.chunk_modality, lay.chunk_unit,
                           10 ** 6, 64)
    n = lay.n_slots
    assert np.array_equal(cp["k"][:n], k)
    assert cp["src_of_dst"][:n].tolist() == list(range(n))
    assert np.array_equal(cp["pos"][:n], lay.pos) and np.array_equal(cp["unit_id"][:n], lay.unit_id)


@pytest.mark.parametrize("seed", range(10))
def test_order_and_rows_vectorised_crosscheck(seed):
    cfg, lay, seg, rng = _case(seed, evict=0.3)
    keep = (rng.random(lay.n_units) < 0.5).astype(np.uint8)
    k, v = storage_np(seg.k_hist), storage_np(seg.v_hist)
    cp = oracle.compact_kv(k, v, lay.unit_id, lay.modality, lay.pos, keep, lay.n_units,
                           storage_np(seg.k_chunk), storage_np(seg.v_chunk), lay.chunk_modality,
                           lay.chunk_unit, 10 ** 6, 64)
    # independent vectorised formulation
    live = lay.unit_id >= 0
    kept_slot = live & (keep[np.maximum(lay.unit_id, 0)] != 0)
    rows = np.flatnonzero(kept_slot)
    deleted_before = np.cumsum(live & ~kept_slot) - (live & ~kept_slot)
    kept = len(rows)
    src = cp["src_of_dst"]
    assert np.all(np.diff(src[:kept]) > 0) and np.array_equal(src[:kept], rows)
    assert np.array_equal(cp["k"][:kept], k[rows]) and np.array_equal(cp["v"][:kept], v[rows])
    assert np.array_equal(cp["pos"][:kept], lay.pos[rows] - deleted_before[rows])
    assert np.array_equal(cp["pos"], np.arange(cp["n_ctx"]))       # dense positions stay dense
    kept_units = np.unique(lay.unit_id[rows])
    assert np.array_equal(cp["unit_id"][:kept], np.searchsorted(kept_units, lay.unit_id[rows]))
    assert cp["n_ctx"] == kept + lay.chunk_len
    assert cp["n_pages"] == -(-cp["n_ctx"] // 64)


def test_capacity_error():
    cfg, lay, seg, _ = _case(7)
    with pytest.raises(CapacityError):
        oracle.compact_kv(storage_np(seg.k_hist), storage_np(seg.v_hist), lay.unit_id,
                          lay.modality, lay.pos, np.ones(lay.n_units, np.uint8), lay.n_units,
                          storage_np(seg.k_chunk), storage_np(seg.v_chunk), lay.chunk_modality,
                          lay.chunk_unit, lay.n_slots + lay.chunk_len - 1, 64)
