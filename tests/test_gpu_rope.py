"""HIP rotary re-encoding in compaction vs the float64 oracle (Applying the retention plan).

Bar: tags, V rows, chunk rows, unrotated dimensions and rows whose position does not change are
bit-exact; every rotated key element is within half a unit in the last place of the storage type
of the exactly rotated value plus 2^-21 of its pair's length (float angle and rotation); with bf16
storage (float arithmetic 16 bits finer than the result) at least 99.9% of them equal the exactly
rotated value rounded to bf16.
"""
import numpy as np
import pytest
import torch

import oracle
import streamgen as sg
from tests._util import storage_np
from tests.test_gpu_parity import dev, gpu_inputs, host, make_step

pytestmark = pytest.mark.gpu

STYLE = {"half": 0, "interleaved": 1}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_34653_amd import omnitide
    omnitide.lib()
    yield


def as_f64(bits, dtype):
    return oracle.to_f64(bits, dtype)


def rounded(x64, dtype):
    t = torch.from_numpy(np.ascontiguousarray(x64)).to(torch.float32)
    if dtype == "bf16":
        return storage_np(t.to(torch.bfloat16))
    return t.numpy()


def ulp(x64, dtype):
    """Spacing of the storage type at |x| (normal range)."""
    mant = 8 if dtype == "bf16" else 24
    e = np.floor(np.log2(np.maximum(np.abs(x64), 1e-30)))
    return np.exp2(e - (mant - 1))


def pair_norm(k64, rot_dims, style):
    a, b = oracle.pair_dims(rot_dims, style)
    n = np.zeros_like(k64)
    r = np.sqrt(k64[..., a] ** 2 + k64[..., b] ** 2)
    n[..., a], n[..., b] = r, r
    return n


def run_rope(cfg, lay, seg, base, rot_dims, style, keep_all=False):
    st = make_step(cfg, lay)
    g = gpu_inputs(lay, [seg])
    st.score(g["k_hist"], g["unit_id"], g["modality"])
    st.select()
    keep = None
    if keep_all:
        keep = torch.ones(lay.n_units, dtype=torch.uint8, device="cuda")
    st.compact(g["k_hist"], g["v_hist"], g["unit_id"], g["modality"], g["pos"], g["k_chunk"],
               g["v_chunk"], g["chunk_modality"], g["chunk_unit"], keep=keep,
               rope=(base, rot_dims, STYLE[style]))
    torch.cuda.synchronize()
    assert int(host(st.d_status)[0]) == 0
    return st


def check(cfg_name, base, rot_dims, style, layout=None):
    cfg = sg.CONFIG_BY_NAME[cfg_name]
    stream = sg.make_stream(cfg)
    lay, seg = stream.layout, stream.segment(0)
    st = run_rope(cfg, lay, seg, base, rot_dims, style)
    k, v = storage_np(seg.k_hist), storage_np(seg.v_hist)
    sc = oracle.score_units(k, cfg.dtype, lay.unit_id, lay.modality, cfg.weights, lay.n_units)
    _, keep, kept = oracle.select_units(sc["wsum"], sc["len"], sc["first"], sc["last"],
                                        sc["flags"], cfg.budget, cfg.recent)
    cp = oracle.compact_kv(k, v, lay.unit_id, lay.modality, lay.pos, keep, lay.n_units,
                           storage_np(seg.k_chunk), storage_np(seg.v_chunk), lay.chunk_modality,
                           lay.chunk_unit, st.cap_dst, cfg.page_size,
                           rope=dict(base=base, dims=rot_dims, style=style, dtype=cfg.dtype))
    n = cp["n_ctx"]
    assert int(host(st.n_ctx)[0]) == n
    for name, key in (("unit_id_dst", "unit_id"), ("modality_dst", "modality"),
                      ("pos_dst", "pos"), ("src_of_dst", "src_of_dst")):
        assert np.array_equal(host(getattr(st, name))[:n], cp[key]), name
    assert np.array_equal(storage_np(st.v_dst[0])[:n], cp["v"])
    got_bits = storage_np(st.k_dst[0])[:n]
    got = as_f64(got_bits, cfg.dtype)
    want = cp["k_f64"]
    src = as_f64(cp["k"], cfg.dtype)
    # exact copies: chunk rows, unshifted rows, dimensions past the rotary width
    shift = np.zeros(n, np.int64)
    shift[:cp["kept"]] = cp["pos"][:cp["kept"]] - np.asarray(lay.pos)[cp["src_of_dst"][:cp["kept"]]]
    assert np.any(shift != 0), "the workload must move some rows"
    same = shift == 0
    assert np.array_equal(got_bits[same], cp["k"][same])
    assert np.array_equal(got_bits[..., rot_dims:], cp["k"][..., rot_dims:])
    # rotated elements
    r = got[~same][..., :rot_dims]
    w = want[~same][..., :rot_dims]
    bound = 0.5 * ulp(w, cfg.dtype) + 2.0 ** -21 * pair_norm(src[~same], rot_dims, style)[..., :rot_dims]
    err = np.abs(r - w)
    assert np.all(err <= bound), float((err - bound).max())
    if cfg.dtype == "bf16":
        exact = rounded(want, cfg.dtype)[~same][..., :rot_dims]
        frac = np.mean(got_bits[~same][..., :rot_dims] == exact)
        assert frac >= 0.999, frac


@pytest.mark.parametrize("cfg_name,base,rot_dims,style", [
    ("single_layer_8k", 1.0e6, 128, "half"),
    ("single_layer_8k", 10000.0, 64, "interleaved"),
    ("tiny_1p6k_f32", 10000.0, 64, "half"),
    ("tiny_1p6k_f32", 500000.0, 48, "interleaved"),
    ("history_80k", 1.0e6, 128, "half"),
])
def test_rope_compaction_parity(cfg_name, base, rot_dims, style):
    check(cfg_name, base, rot_dims, style)


def test_rope_without_deletions_is_plain_copy():
    """Keeping every unit of a pool without holes moves nothing: the result equals the plain
    compaction bit for bit."""
    cfg = sg.CONFIG_BY_NAME["single_layer_8k"]
    stream = sg.make_stream(cfg)
    lay, seg = stream.layout, stream.segment(0)
    live = np.asarray(lay.unit_id) >= 0
    first_hole = np.argmax(~live) if not live.all() else lay.n_slots
    assert first_hole > 0
    st_cap = int(live.sum()) + lay.chunk_len
    st = make_step(cfg, lay, cap_dst=st_cap, budget=int(live.sum()))
    g = gpu_inputs(lay, [seg])
    keep = torch.ones(lay.n_units, dtype=torch.uint8, device="cuda")
    st.score(g["k_hist"], g["unit_id"], g["modality"])
    args = (g["k_hist"], g["v_hist"], g["unit_id"], g["modality"], g["pos"], g["k_chunk"],
            g["v_chunk"], g["chunk_modality"], g["chunk_unit"])
    st.compact(*args, keep=keep)
    torch.cuda.synchronize()
    plain = storage_np(st.k_dst[0]).copy()
    st.compact(*args, keep=keep, rope=(1.0e6, 128, 0))
    torch.cuda.synchronize()
    rot = storage_np(st.k_dst[0])
    n = int(host(st.n_ctx)[0])
    moved = host(st.pos_dst)[:n][: n - lay.chunk_len] != np.asarray(lay.pos)[host(st.src_of_dst)[: n - lay.chunk_len]]
    # rows before the first hole keep their positions and must be copied bit for bit
    rows_same = np.flatnonzero(~moved)
    assert rows_same.size > 0
    assert np.array_equal(rot[rows_same], plain[rows_same])
    assert np.array_equal(rot[n - lay.chunk_len:n], plain[n - lay.chunk_len:n])
