"""The seeded synthetic streams have the sizes and structure the workloads describe."""
import numpy as np
import pytest
import torch

import streamgen as sg

EXPECT = {  # name: (history slots, chunk length, live units)
    "tiny_1p6k_f32": (1634, 89, 37),
    "single_layer_8k": (8192, 665, 28),
    "hires_32k_36layer": (32768, 2329, 32),
    "history_80k": (81920, 665, None),
    "stream_loop_64x665": (16384, 665, None),
}


@pytest.mark.parametrize("cfg", sg.CONFIGS, ids=lambda c: c.name)
def test_structure(cfg):
    st = sg.make_stream(cfg)
    lay = st.layout
    n, L, U = EXPECT[cfg.name]
    assert lay.n_slots == n and lay.chunk_len == L
    if U is not None:
        assert lay.n_units == U
    live = lay.unit_id >= 0
    ids = lay.unit_id[live]
    assert np.all(np.diff(ids) >= 0) and ids[0] == 0 and ids[-1] == lay.n_units - 1
    assert np.array_equal(lay.pos[live], np.arange(live.sum()))
    # text units are 16..64 tokens
    for u in range(lay.n_units):
        m = lay.modality[lay.unit_id == u]
        if m[0] == sg.MOD_TEXT:
            assert 16 <= len(m) <= 64
    if cfg.evict_frac:
        frac = 1 - lay.n_units / lay.n_orig_units
        assert abs(frac - cfg.evict_frac) < 0.01
        assert 50_000 < live.sum() < 65_000


def test_80k_frame_mix():
    lay = sg.make_stream(sg.CONFIG_BY_NAME["history_80k"]).layout
    sizes = np.bincount(lay.orig_unit)
    mods = np.array([lay.modality[lay.orig_unit == u][0] for u in range(lay.n_orig_units)])
    assert sorted(np.unique(sizes[mods == sg.MOD_VIDEO]).tolist()) == [640, 2304]
    assert (sizes[mods == sg.MOD_VIDEO] == 2304).sum() == 14
    assert (mods == sg.MOD_AUDIO).sum() == 375 and sizes[mods == sg.MOD_AUDIO].max() == 25
    assert sizes[mods == sg.MOD_TEXT].sum() == 1249


def test_values_seeded_and_shaped():
    cfg = sg.CONFIG_BY_NAME["single_layer_8k"]
    a = sg.make_stream(cfg).segment(0)
    b = sg.make_stream(cfg).segment(0)
    assert a.k_hist.dtype == torch.bfloat16 and tuple(a.k_hist.shape) == (8192, 8, 128)
    assert tuple(a.q.shape) == (665, 32, 128) and tuple(a.v_chunk.shape) == (665, 8, 128)
    assert torch.equal(a.k_hist, b.k_hist) and torch.equal(a.q, b.q)
    c = sg.make_stream(sg.CONFIG_BY_NAME["hires_32k_36layer"])
    assert not torch.equal(c.segment(0).k_chunk, c.segment(1).k_chunk)
    x = a.k_hist.float()
    assert abs(x.mean().item()) < 0.3 and 0.9 < x.std().item() < 1.3
