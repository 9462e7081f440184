"""Pins of the native-layout oracle: logical eviction, chunk placement, the ordered-suffix cut,
suffix packing and attention over a holey span."""
import json
import os

import numpy as np
import pytest

import oracle


@pytest.fixture(scope="module")
def golden(golden_dir):
    return json.load(open(os.path.join(golden_dir, "native_layout_worked_example.json")))


def test_worked_eviction(golden):
    g = golden
    ev = oracle.evict_logical(g["unit_id"], g["pos"], g["keep_len"], g["n_units"])
    assert ev["unit_id"].tolist() == g["expected_unit_id"]
    assert ev["pos"].tolist() == g["expected_pos"]
    assert ev["unit_remap"].tolist() == g["expected_unit_remap"]
    assert ev["kept"] == g["expected_kept"]
    assert oracle.span_of(ev["unit_id"]) == g["expected_span"]
    assert oracle.active_pages(ev["unit_id"], g["page_size"]) == g["expected_active_pages"]
    c = g["chunk"]
    assert oracle.place_chunk(ev["unit_id"], c["chunk_len"], c["cap"]) == c["expected_slot"]


def test_worked_suffix_cases(golden):
    g = golden
    ev = oracle.evict_logical(g["unit_id"], g["pos"], g["keep_len"], g["n_units"])
    live = ev["unit_id"] >= 0
    n = len(live)
    k = np.arange(n, dtype=np.float64)[:, None, None] * np.ones((1, 1, 2))
    for case in g["suffix_cases"]:
        c, ns = oracle.plan_suffix(live, g["page_size"], case["min_pages"])
        assert (c, ns) == (case["expected_cut"], case["expected_new_span"]), case["min_pages"]
        if c < 0:
            continue
        pk = oracle.pack_suffix(k, -k, ev["unit_id"], np.zeros(n, np.uint8), ev["pos"], c)
        assert pk["moved"] == case["expected_moved"]
        assert pk["unit_id"].tolist() == case["expected_unit_id"]
        assert pk["pos"].tolist() == case["expected_pos"]
        assert oracle.span_of(pk["unit_id"]) == ns
        assert oracle.active_pages(pk["unit_id"], g["page_size"]) == case["expected_active_pages"]
        # every entry's row travelled with it
        for s in np.nonzero(pk["unit_id"] >= 0)[0]:
            src = np.nonzero(ev["pos"] == pk["pos"][s])[0][0]
            assert pk["k"][s, 0, 0] == src and pk["v"][s, 0, 0] == -src


def random_native_pool(rng, n_units, hole_p=0.3):
    """Units as contiguous runs in temporal order with holes between them; dense positions."""
    unit_id, pos = [], []
    p = 0
    for u in range(n_units):
        if rng.random() < hole_p:
            gap = int(rng.integers(1, 9))
            unit_id += [-1] * gap
            pos += [-1] * gap
        n = int(rng.integers(1, 12))
        unit_id += [u] * n
        pos += list(range(p, p + n))
        p += n
    return np.array(unit_id), np.array(pos)


def test_eviction_then_packing_equals_compaction():
    """Logical eviction followed by packing everything equals compacting with the same plan."""
    rng = np.random.default_rng(21)
    for _ in range(60):
        U = int(rng.integers(1, 15))
        uid, pos = random_native_pool(rng, U)
        length = np.bincount(uid[uid >= 0], minlength=U)
        kl = rng.integers(0, length + 2)
        n = len(uid)
        k = rng.standard_normal((n, 2, 4))
        v = rng.standard_normal((n, 2, 4))
        mod = rng.integers(0, 4, n).astype(np.uint8)
        cp = oracle.compact_kv(k, v, uid, mod, pos, None, U, np.zeros((0, 2, 4)),
                               np.zeros((0, 2, 4)), np.zeros(0, np.uint8), np.zeros(0, np.int64),
                               n, 64, keep_len=kl)
        ev = oracle.evict_logical(uid, pos, kl, U)
        assert ev["kept"] == cp["kept"]
        pk = oracle.pack_suffix(k, v, ev["unit_id"], mod, ev["pos"], 0)
        m = cp["kept"]
        assert np.array_equal(pk["unit_id"][:m], cp["unit_id"])
        assert np.array_equal(pk["pos"][:m], cp["pos"])
        assert np.array_equal(pk["k"][:m], cp["k"]) and np.array_equal(pk["v"][:m], cp["v"])
        assert np.array_equal(ev["unit_remap"], cp["unit_remap"])


def test_eviction_rotary_adjustment_equals_compaction():
    """Keys re-rotated at logical eviction (entries in place) equal, row for row, the keys the
    compaction re-encodes for the same plan; evicted and empty slots keep their keys, and a
    unit kept at its old positions (nothing deleted before it) is not rotated."""
    rng = np.random.default_rng(22)
    for trial in range(40):
        U = int(rng.integers(1, 15))
        uid, pos = random_native_pool(rng, U)
        length = np.bincount(uid[uid >= 0], minlength=U)
        kl = rng.integers(0, length + 2)
        n = len(uid)
        k = rng.standard_normal((n, 2, 8)).astype(np.float32)
        rope = dict(base=10000.0, dims=8 if trial % 2 else 4,
                    style="half" if trial % 3 else "interleaved", dtype="f32")
        cp = oracle.compact_kv(k, k, uid, np.ones(n, np.uint8), pos, None, U,
                               np.zeros((0, 2, 8), np.float32), np.zeros((0, 2, 8), np.float32),
                               np.zeros(0, np.uint8), np.zeros(0, np.int64), n, 64, keep_len=kl,
                               rope=rope)
        ev = oracle.evict_logical(uid, pos, kl, U, k=k, rope=rope)
        kept_slots = np.nonzero(ev["unit_id"] >= 0)[0]          # slot order = position order
        assert np.array_equal(ev["k_f64"][kept_slots], cp["k_f64"][:cp["kept"]])
        rest = np.setdiff1d(np.arange(n), kept_slots)
        assert np.array_equal(ev["k_f64"][rest], k[rest].astype(np.float64))
        same = kept_slots[ev["pos"][kept_slots] == pos[kept_slots]]
        assert np.array_equal(ev["k_f64"][same], k[same].astype(np.float64))


def test_suffix_cut_by_exhaustive_packing():
    """The cut equals the largest c whose actual packing (span measured after moving the rows)
    saves the threshold -- not via the closed-form packed span."""
    rng = np.random.default_rng(22)
    for _ in range(150):
        n = int(rng.integers(1, 40))
        live = rng.random(n) < rng.uniform(0.1, 0.9)
        uid = np.where(live, 0, -1)
        P = int(rng.choice([1, 2, 4, 8]))
        T = int(rng.integers(1, 4))
        span = oracle.span_of(uid)
        pages = lambda x: -(-x // P)  # noqa: E731
        want = (-1, span)
        for c in range(0, span + 1):
            pk = oracle.pack_suffix(np.zeros((n, 1, 1)), np.zeros((n, 1, 1)), uid,
                                    np.zeros(n, np.uint8), np.where(live, 0, -1), c)
            ns = oracle.span_of(pk["unit_id"])
            if pages(span) - pages(ns) >= T:
                want = (c, ns)
        assert oracle.plan_suffix(live, P, T) == want


def test_chunk_placement_brute_force():
    rng = np.random.default_rng(23)
    for _ in range(200):
        n = int(rng.integers(0, 30))
        uid = np.where(rng.random(n) < 0.5, 0, -1)
        cap = n + int(rng.integers(0, 6))
        L = int(rng.integers(1, 6))
        occ = np.zeros(cap, bool)
        occ[:n] = uid >= 0
        fits = [s for s in range(cap - L + 1) if not occ[s:s + L].any()]
        if fits:
            assert oracle.place_chunk(uid, L, cap) == fits[0]
        else:
            with pytest.raises(oracle.CapacityError):
                oracle.place_chunk(uid, L, cap)


def gather_by_position(k, v, key_pos):
    """The pool's entries reordered by logical position: the compacted equivalent."""
    idx = np.nonzero(key_pos >= 0)[0]
    idx = idx[np.argsort(key_pos[idx])]
    return k[idx], v[idx]


def test_span_attention_equals_attention_over_the_packed_pool():
    rng = np.random.default_rng(24)
    for trial in range(12):
        U = int(rng.integers(2, 10))
        uid, pos = random_native_pool(rng, U)
        n_hist = int((uid >= 0).sum())
        L = int(rng.integers(1, 6))
        H, G, d = 2, 2, 8
        # scatter the chunk into a random empty run (or the end) and shuffle nothing else
        n = len(uid)
        cap = n + L + 5
        kp = np.full(cap, -1)
        kp[:n] = pos
        uid_c = np.full(cap, -1)
        uid_c[:n] = uid
        s0 = oracle.place_chunk(uid_c, L, cap)
        kp[s0:s0 + L] = n_hist + np.arange(L)
        k = rng.standard_normal((cap, H, d))
        v = rng.standard_normal((cap, H, d))
        k[kp < 0] = np.nan if trial % 2 else 1e30          # empty slots never matter
        v[kp < 0] = np.nan if trial % 2 else -1e30
        q = rng.standard_normal((L, H * G, d))
        span = int(np.nonzero(kp >= 0)[0][-1]) + 1
        got = oracle.span_attention(q, k, v, kp, span, n_hist, 0.3)
        kk, vv = gather_by_position(k, v, kp)
        want = oracle.chunk_attention(q, kk, vv, 0.3)
        assert np.abs(got - want).max() < 1e-12


def test_span_attention_special_cases():
    rng = np.random.default_rng(25)
    d = 4
    k = rng.standard_normal((10, 1, d))
    v = rng.standard_normal((10, 1, d))
    kp = np.full(10, -1)
    kp[7] = 0                                          # a single entry: the query itself
    out = oracle.span_attention(rng.standard_normal((1, 2, d)), k, v, kp, 8, 0, 1.0)
    assert np.array_equal(out[0, 0], v[7, 0]) and np.array_equal(out[0, 1], v[7, 0])
    # identical keys: the mean of the visible values
    k[:] = k[0]
    kp = np.array([3, -1, 0, 1, -1, 2, -1, -1, -1, -1])
    out = oracle.span_attention(rng.standard_normal((2, 1, d)), k, v, kp, 6, 2, 0.5)
    assert np.allclose(out[0, 0], v[[2, 3, 5], 0].mean(axis=0), atol=1e-14)
    assert np.allclose(out[1, 0], v[[0, 2, 3, 5], 0].mean(axis=0), atol=1e-14)
    with pytest.raises(ValueError):
        oracle.span_attention(np.zeros((1, 1, d)), k, v, np.full(10, -1), 10, 0, 1.0)
