"""Pins for the oracle's rotary re-encoding of moved keys (Applying the retention plan).

The reference points are independent of the oracle's real-valued rotation: literal frequencies
and cosines from the rotary-embedding definition, and a complex-exponential formulation of
encoding a raw key at an absolute position.
"""
import numpy as np
import pytest

import oracle
import streamgen as sg


def encode_at(x, pos, base, rot_dims, style):
    """Encode raw keys x [n, H, d] at absolute positions pos [n]: pair j as the complex number
    x_a + i x_b multiplied by exp(i pos theta_j)."""
    x = np.asarray(x, np.float64)
    half = rot_dims // 2
    j = np.arange(half)
    a, b = (j, j + half) if style == "half" else (2 * j, 2 * j + 1)
    theta = np.array([base ** (-(2.0 * t) / rot_dims) for t in range(half)])
    z = (x[..., a] + 1j * x[..., b]) * np.exp(1j * np.outer(pos, theta))[:, None, :]
    out = x.copy()
    out[..., a], out[..., b] = z.real, z.imag
    return out


def test_frequencies_literal():
    th = oracle.rope_thetas(10000.0, 128)
    assert th.shape == (64,)
    assert th[0] == 1.0
    assert th[1] == pytest.approx(0.8659643233600653, rel=1e-15)
    assert th[63] == pytest.approx(1.1547819846894582e-4, rel=1e-13)
    assert oracle.rope_thetas(1.0e6, 64)[32 - 1] == pytest.approx(1.0e6 ** (-62 / 64), rel=1e-15)


@pytest.mark.parametrize("style", ["half", "interleaved"])
def test_unit_vector_rotation(style):
    # a raw key (1, 0) in pair 0 moved by +1 position turns by theta_0 = 1 radian
    k = np.zeros((1, 1, 8))
    a, b = oracle.pair_dims(8, style)
    k[0, 0, a[0]] = 1.0
    r = oracle.shift_keys(k, [1], 10000.0, 8, style)
    assert r[0, 0, a[0]] == pytest.approx(0.5403023058681398, abs=1e-16)
    assert r[0, 0, b[0]] == pytest.approx(0.8414709848078965, abs=1e-16)
    r = oracle.shift_keys(k, [-1], 10000.0, 8, style)
    assert r[0, 0, b[0]] == pytest.approx(-0.8414709848078965, abs=1e-16)


@pytest.mark.parametrize("style", ["half", "interleaved"])
@pytest.mark.parametrize("rot_dims", [128, 64, 32])
def test_shift_equals_encoding_at_new_position(style, rot_dims):
    rng = np.random.default_rng(7)
    n, H, d, base = 40, 3, 128, 10000.0
    x = rng.standard_normal((n, H, d))
    old = np.sort(rng.integers(0, 90000, n))
    new = old - rng.integers(0, 60000, n).clip(max=old)
    stored = encode_at(x, old, base, rot_dims, style)
    moved = oracle.shift_keys(stored, new - old, base, rot_dims, style)
    np.testing.assert_allclose(moved, encode_at(x, new, base, rot_dims, style), rtol=0,
                               atol=1e-9)
    # dimensions past the rotary width are untouched, bit for bit
    assert np.array_equal(moved[..., rot_dims:], stored[..., rot_dims:])


def test_identity_composition_and_norms():
    rng = np.random.default_rng(3)
    k = rng.standard_normal((25, 2, 64))
    assert np.array_equal(oracle.shift_keys(k, np.zeros(25, int), 500000.0, 64, "half"), k)
    s1, s2 = rng.integers(-5000, 5000, 25), rng.integers(-5000, 5000, 25)
    two = oracle.shift_keys(oracle.shift_keys(k, s1, 500000.0, 64, "half"), s2, 500000.0, 64,
                            "half")
    np.testing.assert_allclose(two, oracle.shift_keys(k, s1 + s2, 500000.0, 64, "half"),
                               atol=1e-11)
    a, b = oracle.pair_dims(64, "half")
    r = oracle.shift_keys(k, s1, 500000.0, 64, "half")
    np.testing.assert_allclose(r[..., a] ** 2 + r[..., b] ** 2, k[..., a] ** 2 + k[..., b] ** 2,
                               rtol=1e-12)


def test_compaction_reencodes_history_at_new_positions():
    """End to end: a pool whose keys are encoded at their slot positions, compacted with the
    rotary option, holds every history key encoded at its new position and the chunk as given."""
    cfg = sg.CONFIG_BY_NAME["tiny_1p6k_f32"]
    stream = sg.make_stream(cfg)
    lay = stream.layout
    rng = np.random.default_rng(11)
    H, d = cfg.n_kv_heads, cfg.head_dim
    raw = rng.standard_normal((lay.n_slots, H, d))
    pos = np.asarray(lay.pos, np.int64)
    live = np.asarray(lay.unit_id) >= 0
    enc = np.where(live[:, None, None], encode_at(raw, np.where(live, pos, 0), 10000.0, d, "half"),
                   0.0).astype(np.float32)
    sc = oracle.score_units(enc, "f32", lay.unit_id, lay.modality, cfg.weights, lay.n_units)
    _, keep, kept = oracle.select_units(sc["wsum"], sc["len"], sc["first"], sc["last"],
                                        sc["flags"], cfg.budget, cfg.recent)
    L = lay.chunk_len
    kc = rng.standard_normal((L, H, d)).astype(np.float32)
    cp = oracle.compact_kv(enc, enc, lay.unit_id, lay.modality, lay.pos, keep, lay.n_units, kc,
                           kc, lay.chunk_modality, lay.chunk_unit, cfg.budget + L, cfg.page_size,
                           rope=dict(base=10000.0, dims=d, style="half", dtype="f32"))
    n_hist = cp["kept"]
    assert n_hist == kept and n_hist > 0
    assert np.any(cp["pos"][:n_hist] != pos[cp["src_of_dst"][:n_hist]])   # some rows moved
    want = encode_at(raw[cp["src_of_dst"][:n_hist]], cp["pos"][:n_hist], 10000.0, d, "half")
    # stored keys are float32-rounded encodings, so agreement is to float32 precision
    np.testing.assert_allclose(cp["k_f64"][:n_hist], want, rtol=0, atol=2e-5)
    assert np.array_equal(cp["k_f64"][n_hist:], kc.astype(np.float64))
    assert np.array_equal(cp["k"], np.concatenate([enc[cp["src_of_dst"][:n_hist]], kc]))
