"""Pins for the oracle's unit scoring (closed forms, hand values, invariances, error cases)."""
import math

import numpy as np
import pytest

import oracle
from oracle import TagError
import streamgen as sg
from tests._util import storage_np

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")

# q(x) = floor(min(|x|, 32) * 2^16), worked by hand.
HAND_Q = [
    (0.0, 0), (-0.0, 0), (0.75, 49152), (-1.5, 98304), (31.5, 2064384), (32.0, 2097152),
    (40.0, 2097152), (2.0 ** -16, 1), (2.0 ** -17, 0), (3 * 2.0 ** -17, 1),
    (float("nan"), 2097152), (float("inf"), 2097152), (-float("inf"), 2097152),
    (1e-40, 0), (0.0078125, 512),
]


@pytest.mark.parametrize("x,q", HAND_Q)
def test_quantize_hand_values(x, q):
    assert int(oracle.quantize_magnitude(np.array([x]))[0]) == q


def test_weights_exact_q88():
    assert oracle.weights_q88((2.0, 1.0, 1.5, 2.0)).tolist() == [512, 256, 384, 512]
    with pytest.raises(ValueError):
        oracle.weights_q88((1.0, 1.0, 1.0 / 3.0, 1.0))
    with pytest.raises(ValueError):
        oracle.weights_q88((1.0, 0.0, 1.0, 1.0))
    with pytest.raises(ValueError):
        oracle.weights_q88((1.0, 5.0, 1.0, 1.0))


def _const_case(c, dtype):
    # units: video 3 slots, audio 2 slots, text 4 slots, H=2, d=8
    unit_id = np.array([0, 0, 0, 1, 1, 2, 2, 2, 2], np.int32)
    mod = np.array([1, 1, 1, 2, 2, 3, 3, 3, 3], np.uint8)
    k = np.full((9, 2, 8), c, np.float32)
    if dtype == "bf16":
        import torch
        k = storage_np(torch.from_numpy(k).to(torch.bfloat16))
    return k, unit_id, mod


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("c,qc", [(0.75, 49152), (-1.5, 98304), (40.0, 2097152), (2.0 ** -17, 0)])
def test_closed_form_constant_keys(dtype, c, qc):
    k, unit_id, mod = _const_case(c, dtype)
    sc = oracle.score_units(k, dtype, unit_id, mod, sg.DEFAULT_WEIGHTS, 3)
    a = 16 * qc                              # H*d elements per slot
    assert sc["wsum"].tolist() == [256 * a * 3, 384 * a * 2, 512 * a * 4]
    assert sc["len"].tolist() == [3, 2, 4]
    assert sc["first"].tolist() == [0, 3, 5] and sc["last"].tolist() == [2, 4, 8]
    assert sc["flags"].tolist() == [0, 0, 0]


def test_nan_inf_count_as_clamp():
    k, unit_id, mod = _const_case(0.0, "f32")
    k[0, 0, 0] = np.nan
    k[4, 1, 7] = -np.inf
    sc = oracle.score_units(k, "f32", unit_id, mod, sg.DEFAULT_WEIGHTS, 3)
    assert sc["wsum"].tolist() == [256 * 2097152, 384 * 2097152, 0]


def test_holes_and_structure_fields():
    unit_id = np.array([-1, 0, 0, -1, -1, 1, 2, 2, -1], np.int32)
    mod = np.array([1, 0, 3, 1, 1, 2, 1, 1, 1], np.uint8)
    rng = np.random.default_rng(0)
    k = rng.standard_normal((9, 1, 4)).astype(np.float32)
    k_big = k.copy()
    k_big[unit_id < 0] = 1e30            # hole contents never matter
    sc = oracle.score_units(k, "f32", unit_id, mod, sg.DEFAULT_WEIGHTS, 4)
    sc2 = oracle.score_units(k_big, "f32", unit_id, mod, sg.DEFAULT_WEIGHTS, 4)
    assert all(np.array_equal(sc[f], sc2[f]) for f in sc)
    assert sc["len"].tolist() == [2, 1, 2, 0]
    assert sc["first"].tolist() == [1, 5, 6, 9]      # empty unit: n_slots
    assert sc["last"].tolist() == [2, 5, 7, -1]      # empty unit: -1
    assert sc["flags"].tolist() == [1, 0, 0, 0]
    assert sc["wsum"][3] == 0


def test_sign_and_permutation_invariance():
    cfg, lay, seg = sg.custom_stream([(1, 7), (2, 5), (3, 9)], [(1, 3)], dtype="bf16",
                                     n_kv_heads=2, head_dim=64)
    k = storage_np(seg.k_hist)
    base = oracle.score_units(k, "bf16", lay.unit_id, lay.modality, cfg.weights, lay.n_units)
    neg = k ^ np.uint16(0x8000)                    # flip every sign bit
    sc = oracle.score_units(neg, "bf16", lay.unit_id, lay.modality, cfg.weights, lay.n_units)
    assert np.array_equal(base["wsum"], sc["wsum"])
    perm = np.concatenate([np.random.default_rng(1).permutation(7), 7 + np.arange(14)])
    sc = oracle.score_units(k[perm], "bf16", lay.unit_id, lay.modality, cfg.weights, lay.n_units)
    assert np.array_equal(base["wsum"], sc["wsum"])


def test_modality_weight_ratio():
    # identical keys tagged video, audio, text, marker: sums in ratio 256 : 384 : 512 : 512
    rng = np.random.default_rng(3)
    row = rng.standard_normal((1, 2, 8)).astype(np.float32)
    k = np.repeat(row, 4, axis=0)
    sc = oracle.score_units(k, "f32", np.array([0, 1, 2, 3], np.int32),
                            np.array([1, 2, 3, 4], np.uint8), (1.0, 1.0, 1.5, 2.5), 4)
    w = sc["wsum"]
    assert w[0] * 384 == w[1] * 256 and w[0] * 640 == w[2] * 256 and w[3] == w[2]


def test_mixed_unit_closed_form():
    """One grammar unit (markers, 3 video, 2 audio, 1 text) of constant keys c = 0.75:
    a_s = 16 * 49152 per slot, W = a_s * (6 markers * 512 + 3 * 256 + 2 * 384 + 512)."""
    lay = sg.build_layout([sg.grammar_unit(3, 2, 1)], [])
    n = lay.n_slots
    assert n == 12 and (lay.modality == 4).sum() == 6
    k = np.full((n, 2, 8), 0.75, np.float32)
    sc = oracle.score_units(k, "f32", lay.unit_id, lay.modality, sg.DEFAULT_WEIGHTS, 1)
    a = 16 * 49152
    assert sc["wsum"].tolist() == [a * (6 * 512 + 3 * 256 + 2 * 384 + 512)]
    assert sc["len"].tolist() == [12] and sc["flags"].tolist() == [0]


def test_brute_force_tiny_config():
    """Per-element scalar loop (math.floor on Python floats) on a small slice of the 1.6K case."""
    st = sg.make_stream(sg.CONFIG_BY_NAME["tiny_1p6k_f32"])
    seg = st.segment(0)
    n = 200
    k = storage_np(seg.k_hist)[:n]
    uid = st.layout.unit_id[:n]
    mod = st.layout.modality[:n]
    U = int(uid.max()) + 1
    sc = oracle.score_units(k, "f32", uid, mod, sg.DEFAULT_WEIGHTS, U)
    wq = {0: 512, 1: 256, 2: 384, 3: 512}
    expect = [0] * U
    for s in range(n):
        tot = 0
        for x in k[s].reshape(-1).tolist():
            ax = abs(x)
            tot += math.floor((32.0 if (ax != ax or ax > 32.0) else ax) * 65536.0)
        expect[uid[s]] += wq[int(mod[s])] * tot
    assert sc["wsum"].tolist() == expect


@pytest.mark.parametrize("bad", ["id_high", "id_low", "mod"])
def test_tag_errors(bad):
    unit_id = np.array([0, 0, 1], np.int32)
    mod = np.array([1, 1, 2], np.uint8)
    if bad == "id_high":
        unit_id[2] = 2
    elif bad == "id_low":
        unit_id[0] = -2
    else:
        mod[1] = 5
    with pytest.raises(TagError):
        oracle.score_units(np.zeros((3, 1, 4), np.float32), "f32", unit_id, mod,
                           sg.DEFAULT_WEIGHTS, 2)
