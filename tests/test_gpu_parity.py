"""HIP path vs the CPU oracle, through the C ABI (ctypes binding).

Bar: score, selection and compaction bit-exact (integers and raw KV bytes); attention within
max |err| <= 1e-2 and mean |err| <= 1e-3 of the float64 oracle on the same bf16 inputs, on every
query row (the mean over the whole output), full-size workloads included.
"""
import concurrent.futures as cf
import types

import numpy as np
import pytest
import torch

import oracle
import streamgen as sg
from tests._util import storage_np

pytestmark = pytest.mark.gpu

MAX_ABS, MEAN_ABS = 1e-2, 1e-3


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_34653_amd import omnitide
    omnitide.lib()
    yield


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    return t.detach().cpu().numpy()


def make_step(cfg, lay, n_seg=1, cap_dst=None, n_units=None, budget=None, recent=None):
    from paper_2609_34653_amd.step import StreamStep
    return StreamStep(n_seg=n_seg, n_slots=lay.n_slots, n_units=n_units or lay.n_units,
                      n_q_heads=cfg.n_q_heads, n_kv_heads=cfg.n_kv_heads, head_dim=cfg.head_dim,
                      chunk_len=lay.chunk_len, budget=cfg.budget if budget is None else budget,
                      recent=cfg.recent if recent is None else recent, page_size=cfg.page_size,
                      weights=cfg.weights,
                      kv_dtype=torch.bfloat16 if cfg.dtype == "bf16" else torch.float32,
                      cap_dst=cap_dst)


def gpu_inputs(lay, segs):
    n = len(segs)
    return dict(
        k_hist=torch.stack([s.k_hist for s in segs]).cuda(),
        v_hist=torch.stack([s.v_hist for s in segs]).cuda(),
        unit_id=dev(np.tile(lay.unit_id, n)), modality=dev(np.tile(lay.modality, n)),
        pos=dev(np.tile(lay.pos, n)),
        k_chunk=torch.stack([s.k_chunk for s in segs]).cuda(),
        v_chunk=torch.stack([s.v_chunk for s in segs]).cuda(),
        chunk_modality=dev(lay.chunk_modality), chunk_unit=dev(lay.chunk_unit),
        q=torch.stack([s.q for s in segs]).cuda())


def run_gpu(cfg, st, inp, attend=True, sync=True):
    st.score(inp["k_hist"], inp["unit_id"], inp["modality"])
    st.select()
    st.compact(inp["k_hist"], inp["v_hist"], inp["unit_id"], inp["modality"], inp["pos"],
               inp["k_chunk"], inp["v_chunk"], inp["chunk_modality"], inp["chunk_unit"])
    if attend:   # float32 pools: the library rounds q, k, v to bf16 (nearest even) itself
        st.attend(inp["q"], cfg.scale)
    if sync:
        torch.cuda.synchronize()


def check_segment(cfg, lay, seg, st, si, n_units=None):
    """Compare segment si of the GPU step with the oracle; returns the oracle's compaction."""
    U = n_units or lay.n_units
    sl = slice(si * U, (si + 1) * U)
    k = storage_np(seg.k_hist)
    sc = oracle.score_units(k, cfg.dtype, lay.unit_id, lay.modality, cfg.weights, U)
    assert np.array_equal(host(st.unit_wsum)[sl], sc["wsum"])
    assert np.array_equal(host(st.unit_len)[sl], sc["len"])
    assert np.array_equal(host(st.unit_first)[sl], sc["first"])
    assert np.array_equal(host(st.unit_last)[sl], sc["last"])
    assert np.array_equal(host(st.unit_flags)[sl], sc["flags"])
    score, keep, kept = oracle.select_units(sc["wsum"], sc["len"], sc["first"], sc["last"],
                                            sc["flags"], st.budget, st.recent)
    assert np.array_equal(host(st.unit_score)[sl], score)
    assert np.array_equal(host(st.keep)[sl], keep)
    assert int(host(st.kept_tokens)[si]) == kept
    cp = oracle.compact_kv(k, storage_np(seg.v_hist), lay.unit_id, lay.modality, lay.pos, keep, U,
                           storage_np(seg.k_chunk), storage_np(seg.v_chunk), lay.chunk_modality,
                           lay.chunk_unit, st.cap_dst, st.page_size)
    n = cp["n_ctx"]
    assert int(host(st.n_ctx)[si]) == n and int(host(st.n_pages)[si]) == cp["n_pages"]
    kd = storage_np(st.k_dst[si])
    vd = storage_np(st.v_dst[si])
    assert np.array_equal(kd[:n], cp["k"]) and np.array_equal(vd[:n], cp["v"])
    cap = st.cap_dst
    tags = slice(si * cap, (si + 1) * cap)
    uid = host(st.unit_id_dst)[tags]
    assert np.array_equal(uid[:n], cp["unit_id"]) and np.all(uid[n:] == -1)
    assert np.array_equal(host(st.modality_dst)[tags][:n], cp["modality"])
    assert np.array_equal(host(st.pos_dst)[tags][:n], cp["pos"])
    assert np.array_equal(host(st.src_of_dst)[tags][:n], cp["src_of_dst"])
    assert np.all(host(st.src_of_dst)[tags][n:] == -1)
    assert np.array_equal(host(st.unit_remap)[sl], cp["unit_remap"])
    return cp


def check_attention(cfg, lay, seg, st, si, cp, rows=None):
    """Oracle rows (all, or the positions ``rows``) vs GPU output of segment si; the mean
    absolute error is taken over everything compared."""
    to64 = lambda a: oracle.to_f64(a, "bf16")   # noqa: E731
    qb = storage_np(seg.q.to(torch.bfloat16)) if cfg.dtype == "f32" else storage_np(seg.q)
    if cfg.dtype == "f32":
        kb = storage_np(torch.from_numpy(cp["k"]).to(torch.bfloat16))
        vb = storage_np(torch.from_numpy(cp["v"]).to(torch.bfloat16))
    else:
        kb, vb = cp["k"], cp["v"]
    out = host(st.out[si])
    L = lay.chunk_len
    kept = cp["n_ctx"] - L
    q64, k64, v64 = to64(qb), to64(kb), to64(vb)
    if rows is None:
        ref = oracle.chunk_attention(q64, k64, v64, cfg.scale)
        got = out
    else:
        ref = np.stack([oracle.chunk_attention(q64[i:i + 1], k64[:kept + i + 1],
                                               v64[:kept + i + 1], cfg.scale)[0]
                        for i in rows])
        got = out[rows]
    err = np.abs(got.astype(np.float64) - ref)
    assert np.isfinite(got).all()
    assert err.max() <= MAX_ABS, err.max()
    assert err.mean() <= MEAN_ABS, err.mean()
    return err.max(), err.mean()


@pytest.mark.parametrize("name", ["tiny_1p6k_f32", "single_layer_8k", "history_80k"])
def test_step_parity(name):
    """Every output of the step; attention compared on every query row, mean over all."""
    cfg = sg.CONFIG_BY_NAME[name]
    stream = sg.make_stream(cfg)
    lay, seg = stream.layout, stream.segment(0)
    st = make_step(cfg, lay)
    run_gpu(cfg, st, gpu_inputs(lay, [seg]))
    assert int(host(st.d_status)[0]) == 0
    cp = check_segment(cfg, lay, seg, st, 0)
    check_attention(cfg, lay, seg, st, 0, cp)


HIRES_ATTN_LAYERS = (0, 17, 35)


@pytest.fixture(scope="module")
def hires36():
    """The 32K high-resolution workload as the benchmark launches it: all 36 layers in one
    36-segment call of each entry point (host-generated layers, one seed per layer).  Returns
    the host generator's layers and a host copy of every output."""
    cfg = sg.CONFIG_BY_NAME["hires_32k_36layer"]
    stream = sg.make_stream(cfg)
    lay = stream.layout
    with cf.ThreadPoolExecutor(12) as ex:
        segs = list(ex.map(stream.segment, range(cfg.n_layers)))
    st = make_step(cfg, lay, n_seg=cfg.n_layers)
    run_gpu(cfg, st, gpu_inputs(lay, segs))
    assert int(host(st.d_status)[0]) == 0
    names = ("unit_wsum", "unit_len", "unit_first", "unit_last", "unit_flags", "unit_score",
             "keep", "kept_tokens", "n_ctx", "n_pages", "k_dst", "v_dst", "unit_id_dst",
             "modality_dst", "pos_dst", "src_of_dst", "unit_remap", "out")
    snap = types.SimpleNamespace(**{n: getattr(st, n).cpu() for n in names},
                                 budget=st.budget, recent=st.recent, cap_dst=st.cap_dst,
                                 page_size=st.page_size)
    del st
    torch.cuda.empty_cache()
    return cfg, lay, segs, snap


@pytest.mark.parametrize("group", range(4))
def test_hires_36_layers_bit_exact(hires36, group):
    """Score, select and compaction of nine of the 36 layers, bit-exact (raw KV bytes, every
    tag)."""
    cfg, lay, segs, snap = hires36
    layers = range(9 * group, 9 * group + 9)
    with cf.ThreadPoolExecutor(9) as ex:
        list(ex.map(lambda i: check_segment(cfg, lay, segs[i], snap, i), layers))


@pytest.mark.parametrize("layer", HIRES_ATTN_LAYERS)
def test_hires_36_layers_attention(hires36, layer):
    """All 2,329 query rows of three layers of the 36-segment call."""
    cfg, lay, segs, snap = hires36
    cp = check_segment(cfg, lay, segs[layer], snap, layer)
    check_attention(cfg, lay, segs[layer], snap, layer, cp)


def test_stream_loop_chained_steps():
    """All 64 stream-loop steps chained on the device: each step's destination pool is the next
    step's source (no host sync).  Score, select and compaction bit-exact at every step against
    the oracle chained on its own outputs; attention on every query row every 8th step."""
    from paper_2609_34653_amd.step import StreamStep
    cfg = sg.CONFIG_BY_NAME["stream_loop_64x665"]
    stream = sg.make_stream(cfg)
    lay, seg0 = stream.layout, stream.segment(0)
    U = 512
    cap = cfg.budget + lay.chunk_len
    # GPU chain
    src = dict(k=seg0.k_hist.cuda()[None], v=seg0.v_hist.cuda()[None], uid=dev(lay.unit_id),
               mod=dev(lay.modality), pos=dev(lay.pos))
    o_k, o_v = storage_np(seg0.k_hist), storage_np(seg0.v_hist)
    o_uid, o_mod, o_pos = lay.unit_id.astype(np.int64), lay.modality, lay.pos
    for t in range(cfg.steps):
        clay, cseg = sg.loop_chunk(cfg, t)
        n_slots = src["k"].shape[1]
        st = StreamStep(n_seg=1, n_slots=n_slots, n_units=U, n_q_heads=cfg.n_q_heads,
                        n_kv_heads=cfg.n_kv_heads, head_dim=cfg.head_dim,
                        chunk_len=clay.chunk_len, budget=cfg.budget, recent=cfg.recent,
                        page_size=cfg.page_size, weights=cfg.weights, cap_dst=cap)
        st.score(src["k"], src["uid"], src["mod"])
        st.select()
        st.compact(src["k"], src["v"], src["uid"], src["mod"], src["pos"], cseg.k_chunk.cuda()[None],
                   cseg.v_chunk.cuda()[None], dev(clay.chunk_modality), dev(clay.chunk_unit))
        st.attend(cseg.q.cuda()[None], cfg.scale)
        torch.cuda.synchronize()
        assert int(host(st.d_status)[0]) == 0, t
        # oracle chain on the same state
        sc = oracle.score_units(o_k, "bf16", o_uid, o_mod, cfg.weights, U)
        for key, name in (("wsum", "unit_wsum"), ("len", "unit_len"), ("first", "unit_first"),
                          ("last", "unit_last"), ("flags", "unit_flags")):
            assert np.array_equal(host(getattr(st, name)), sc[key]), (t, key)
        score, keep, kept = oracle.select_units(sc["wsum"], sc["len"], sc["first"], sc["last"],
                                                sc["flags"], cfg.budget, cfg.recent)
        assert np.array_equal(host(st.unit_score), score), t
        assert np.array_equal(host(st.keep), keep) and int(host(st.kept_tokens)[0]) == kept, t
        cp = oracle.compact_kv(o_k, o_v, o_uid, o_mod, o_pos, keep, U, storage_np(cseg.k_chunk),
                               storage_np(cseg.v_chunk), clay.chunk_modality, clay.chunk_unit,
                               cap, cfg.page_size)
        n = cp["n_ctx"]
        assert int(host(st.n_ctx)[0]) == n and int(host(st.n_pages)[0]) == cp["n_pages"], t
        assert np.array_equal(storage_np(st.k_dst[0])[:n], cp["k"]), t
        assert np.array_equal(storage_np(st.v_dst[0])[:n], cp["v"]), t
        for key, name in (("unit_id", "unit_id_dst"), ("modality", "modality_dst"),
                          ("pos", "pos_dst"), ("src_of_dst", "src_of_dst")):
            assert np.array_equal(host(getattr(st, name))[:n], cp[key]), (t, key)
        assert np.all(host(st.unit_id_dst)[n:] == -1) and np.all(host(st.pos_dst)[n:] == -1)
        assert np.array_equal(host(st.unit_remap), cp["unit_remap"]), t
        # Whole units stop at the first misfit, so the history kept is at most the budget
        # (usually less), and the pool holds it plus the whole chunk.
        assert kept <= cfg.budget and n == kept + clay.chunk_len, t
        if t % 8 == 7:
            check_attention(cfg, clay, cseg, st, 0, cp)
        # next state: the destination pool with its empty tail
        pad = cap - n
        tail = np.zeros((pad,) + cp["k"].shape[1:], cp["k"].dtype)   # empty slots
        o_k = np.concatenate([cp["k"], tail])
        o_v = np.concatenate([cp["v"], tail])
        o_uid = np.concatenate([cp["unit_id"], np.full(pad, -1)])
        o_mod = np.concatenate([cp["modality"], np.zeros(pad, np.int64)]).astype(np.uint8)
        o_pos = np.concatenate([cp["pos"], np.full(pad, -1)])
        src = dict(k=st.k_dst, v=st.v_dst, uid=st.unit_id_dst, mod=st.modality_dst,
                   pos=st.pos_dst)
        keep_alive = st  # noqa: F841  (buffers of this step feed the next)


# ----------------------------------------------------------------------------- edge cases

def _custom(units, chunk, **kw):
    return sg.custom_stream(units, chunk, **kw)


def _run_custom(cfg, lay, seg, **kw):
    st = make_step(cfg, lay, **kw)
    run_gpu(cfg, st, gpu_inputs(lay, [seg]))
    return st


@pytest.mark.parametrize("budget,recent", [(0, 0), (5, 0), (10 ** 6, 3)])
def test_budget_extremes(budget, recent):
    units = [(1, 64), (2, 25), (3, 17), (1, 64), (2, 25), (1, 3)]
    cfg, lay, seg = _custom(units, [(1, 37), (2, 5)], n_q_heads=8, n_kv_heads=2, head_dim=128,
                            budget=budget, recent=recent)
    st = _run_custom(cfg, lay, seg)
    assert int(host(st.d_status)[0]) == 0
    cp = check_segment(cfg, lay, seg, st, 0)
    check_attention(cfg, lay, seg, st, 0, cp)


def test_single_query_no_history_returns_value():
    cfg, lay, seg = _custom([(1, 5)], [(2, 1)], n_q_heads=4, n_kv_heads=1, head_dim=64,
                            budget=0, recent=0)
    st = _run_custom(cfg, lay, seg)
    out = host(st.out[0, 0])                                    # [Hq, d]
    v0 = oracle.to_f64(storage_np(seg.v_chunk), "bf16")[0, 0]
    assert np.abs(out - v0[None, :]).max() < 1e-6


def test_holes_on_page_edges_and_units_across_tiles():
    rng = np.random.default_rng(5)
    units = sg.random_units(rng, 60, lo=1, hi=70)
    evicted = {1, 2, 7, 8, 9, 20, 33, 34, 50}
    cfg, lay, seg = _custom(units, [(1, 70), (3, 9)], n_q_heads=16, n_kv_heads=4, head_dim=128,
                            budget=700, recent=79, evicted=evicted, page_size=32)
    st = _run_custom(cfg, lay, seg)
    assert int(host(st.d_status)[0]) == 0
    cp = check_segment(cfg, lay, seg, st, 0)
    check_attention(cfg, lay, seg, st, 0, cp)


def test_system_prefix_protected_and_over_budget():
    units = [(0, 40), (1, 64), (2, 25), (3, 30), (1, 64)]
    cfg, lay, seg = _custom(units, [(1, 16)], budget=100, recent=30, head_dim=64)
    st = _run_custom(cfg, lay, seg)
    assert int(host(st.d_status)[0]) == 0
    assert host(st.keep)[0] == 1
    check_segment(cfg, lay, seg, st, 0)
    cfg2, lay2, seg2 = _custom(units, [(1, 16)], budget=39, recent=30, head_dim=64)
    st2 = make_step(cfg2, lay2)
    inp = gpu_inputs(lay2, [seg2])
    st2.score(inp["k_hist"], inp["unit_id"], inp["modality"])
    st2.select()
    torch.cuda.synchronize()
    assert int(host(st2.d_status)[0]) == oracle.BudgetError.code
    assert host(st2.keep).sum() == 0 and int(host(st2.kept_tokens)[0]) == 0


def test_tag_errors_reported():
    cfg, lay, seg = _custom([(1, 10), (2, 10), (3, 10)], [(1, 4)], head_dim=64)
    for case in ("modality", "unit_range", "split_unit"):
        uid = lay.unit_id.copy()
        mod = lay.modality.copy()
        if case == "modality":
            mod[3] = 7
        elif case == "unit_range":
            uid[4] = 3
        else:
            uid[12] = 2        # unit 1 broken into two runs around a unit-2 slot
        st = make_step(cfg, lay)
        k = seg.k_hist.cuda()
        st.score(k, dev(uid), dev(mod))
        st.select()
        torch.cuda.synchronize()
        assert int(host(st.d_status)[0]) == oracle.TagError.code, case


def test_capacity_error_on_device():
    cfg, lay, seg = _custom([(1, 50), (2, 50)], [(1, 20)], head_dim=64, budget=100, recent=0)
    st = make_step(cfg, lay, cap_dst=60)
    inp = gpu_inputs(lay, [seg])
    st.score(inp["k_hist"], inp["unit_id"], inp["modality"])
    st.compact(inp["k_hist"], inp["v_hist"], inp["unit_id"], inp["modality"], inp["pos"],
               inp["k_chunk"], inp["v_chunk"], inp["chunk_modality"], inp["chunk_unit"],
               keep=torch.ones(lay.n_units, dtype=torch.uint8, device="cuda"))
    torch.cuda.synchronize()
    assert int(host(st.d_status)[0]) == oracle.CapacityError.code
    assert int(host(st.n_ctx)[0]) == 0 and np.all(host(st.unit_id_dst) == -1)


def test_empty_chunk_compaction():
    from paper_2609_34653_amd import omnitide as ot
    cfg, lay, seg = _custom([(1, 40), (2, 25), (3, 9)], [(1, 4)], head_dim=64, budget=50,
                            recent=9)
    st = make_step(cfg, lay)
    inp = gpu_inputs(lay, [seg])
    st.score(inp["k_hist"], inp["unit_id"], inp["modality"])
    st.select()
    ot.omnitide_compact_kv(inp["k_hist"], inp["v_hist"], cfg.page_size, inp["unit_id"],
                           inp["modality"], inp["pos"], st.keep, st.unit_len, st.unit_first,
                           lay.n_units, None, None, None, None, st.k_dst, st.v_dst,
                           st.unit_id_dst, st.modality_dst, st.pos_dst, st.src_of_dst,
                           st.unit_remap, st.n_ctx, st.n_pages, st.compact_ws, st.d_status)
    torch.cuda.synchronize()
    sc = oracle.score_units(storage_np(seg.k_hist), "bf16", lay.unit_id, lay.modality,
                            cfg.weights, lay.n_units)
    _, keep, kept = oracle.select_units(sc["wsum"], sc["len"], sc["first"], sc["last"],
                                        sc["flags"], 50, 9)
    cp = oracle.compact_kv(storage_np(seg.k_hist), storage_np(seg.v_hist), lay.unit_id,
                           lay.modality, lay.pos, keep, lay.n_units, np.zeros((0, 1, 64), np.uint16),
                           np.zeros((0, 1, 64), np.uint16), np.zeros(0, np.uint8),
                           np.zeros(0, np.int32), st.cap_dst, cfg.page_size)
    assert int(host(st.n_ctx)[0]) == cp["n_ctx"] == kept
    assert np.array_equal(storage_np(st.k_dst[0])[:kept], cp["k"])


@pytest.mark.parametrize("U", [1, 2, 8192])
def test_select_unit_count_extremes(U):
    from paper_2609_34653_amd import omnitide as ot
    rng = np.random.default_rng(U)
    lens = rng.integers(0, 6, size=U)
    first = np.zeros(U, np.int64)
    last = np.zeros(U, np.int64)
    s = 0
    for u in range(U):
        first[u], last[u] = (s, s + lens[u] - 1) if lens[u] else (10 ** 6, -1)
        s += lens[u]
    wsum = lens * rng.integers(0, 50, size=U) * 1000 + rng.integers(0, 3, size=U)
    flags = (rng.random(U) < 0.01).astype(np.int64)
    budget = int(lens.sum() * 0.6) + int(lens[flags == 1].sum())
    score, keep, kept = oracle.select_units(wsum, lens, first, last, flags, budget, 20)
    i32 = lambda a: dev(np.asarray(a, np.int32))   # noqa: E731
    sc_d = torch.zeros(U, dtype=torch.int64, device="cuda")
    keep_d = torch.zeros(U, dtype=torch.uint8, device="cuda")
    kept_d = torch.zeros(1, dtype=torch.int32, device="cuda")
    stat = torch.zeros(1, dtype=torch.int32, device="cuda")
    ot.omnitide_select_units(dev(wsum.astype(np.int64)), i32(lens), i32(first), i32(last),
                             i32(flags), 1, U, budget, 20, sc_d, keep_d, kept_d, stat)
    torch.cuda.synchronize()
    assert int(host(stat)[0]) == 0
    assert np.array_equal(host(sc_d), score) and np.array_equal(host(keep_d), keep)
    assert int(host(kept_d)[0]) == kept


def test_determinism_and_untouched_tail():
    cfg = sg.CONFIG_BY_NAME["single_layer_8k"]
    stream = sg.make_stream(cfg)
    lay, seg = stream.layout, stream.segment(0)
    inp = gpu_inputs(lay, [seg])
    st = make_step(cfg, lay)
    st.k_dst.view(torch.int16).fill_(-1)       # 0xFFFF poison
    st.v_dst.view(torch.int16).fill_(-1)
    run_gpu(cfg, st, inp)
    first = (host(st.unit_wsum).copy(), host(st.out).copy(), storage_np(st.k_dst).copy())
    n = int(host(st.n_ctx)[0])
    assert np.all(first[2][0, n:] == 0xFFFF)
    run_gpu(cfg, st, inp)
    assert np.array_equal(host(st.unit_wsum), first[0])
    assert np.array_equal(host(st.out), first[1])
    assert np.array_equal(storage_np(st.k_dst), first[2])


def test_full_budget_matches_uncompacted_attention_bitwise():
    """With every unit kept and no holes, compaction is the identity, so attention over the
    compacted pool equals the same kernel over [history || chunk] laid out directly."""
    units = [(1, 200), (2, 25), (3, 40), (1, 200), (2, 25)]
    cfg, lay, seg = _custom(units, [(1, 120), (2, 25)], n_q_heads=32, n_kv_heads=8,
                            head_dim=128, budget=10 ** 5, recent=145)
    st = _run_custom(cfg, lay, seg)
    assert host(st.keep).all()
    n = lay.n_slots + lay.chunk_len
    cap = st.cap_dst
    k_all = torch.zeros(1, cap, 8, 128, dtype=torch.bfloat16, device="cuda")
    v_all = torch.zeros_like(k_all)
    k_all[0, :n] = torch.cat([seg.k_hist, seg.k_chunk]).cuda()
    v_all[0, :n] = torch.cat([seg.v_hist, seg.v_chunk]).cuda()
    assert torch.equal(k_all[0, :n], st.k_dst[0, :n])
    from paper_2609_34653_amd import omnitide as ot
    out2 = torch.zeros_like(st.out)
    nctx = torch.tensor([n], dtype=torch.int32, device="cuda")
    ot.omnitide_chunk_attn(seg.q.cuda()[None], k_all, v_all, nctx, cfg.scale, out2, st.attn_ws)
    torch.cuda.synchronize()
    assert torch.equal(out2, st.out)


def _random_plans(rng, n_seg, U, tie_levels):
    lens = rng.integers(0, 40, size=(n_seg, U))
    first = np.zeros((n_seg, U), np.int64)
    last = np.zeros((n_seg, U), np.int64)
    for si in range(n_seg):
        s = 0
        for u in range(U):
            first[si, u], last[si, u] = (s, s + lens[si, u] - 1) if lens[si, u] else (10 ** 6, -1)
            s += lens[si, u]
    wsum = lens * rng.integers(0, tie_levels, size=(n_seg, U)) * 977 \
        + rng.integers(0, 5, size=(n_seg, U)) * (tie_levels > 4)
    flags = (rng.random((n_seg, U)) < 0.02).astype(np.int64)
    return lens, first, last, wsum, flags


@pytest.mark.parametrize("U,tie_levels", [(500, 3), (512, 1000000), (37, 2), (600, 4), (1500, 10 ** 6)])
def test_select_random_instances_many_segments(U, tie_levels):
    """Many random plans in one multi-segment call: heavy ties, empty units, system units."""
    from paper_2609_34653_amd import omnitide as ot
    rng = np.random.default_rng(U * 7 + tie_levels % 97)
    n_seg = 48
    lens, first, last, wsum, flags = _random_plans(rng, n_seg, U, tie_levels)
    budget = int(np.median(lens.sum(1)) * 0.5)
    recent = 60
    i32 = lambda a: dev(np.asarray(a, np.int32).reshape(-1))   # noqa: E731
    sc_d = torch.zeros(n_seg * U, dtype=torch.int64, device="cuda")
    keep_d = torch.zeros(n_seg * U, dtype=torch.uint8, device="cuda")
    kept_d = torch.zeros(n_seg, dtype=torch.int32, device="cuda")
    stat = torch.zeros(1, dtype=torch.int32, device="cuda")
    flags[:, :] = np.where((lens * flags).sum(1, keepdims=True) > budget, 0, flags)
    ot.omnitide_select_units(dev(wsum.astype(np.int64).reshape(-1)), i32(lens), i32(first),
                             i32(last), i32(flags), n_seg, U, budget, recent, sc_d, keep_d, kept_d,
                             stat)
    torch.cuda.synchronize()
    assert int(host(stat)[0]) == 0
    keep_h, sc_h, kept_h = host(keep_d).reshape(n_seg, U), host(sc_d).reshape(n_seg, U), host(kept_d)
    for si in range(n_seg):
        score, keep, kept = oracle.select_units(wsum[si], lens[si], first[si], last[si],
                                                flags[si], budget, recent)
        assert np.array_equal(sc_h[si], score)
        assert np.array_equal(keep_h[si], keep), si
        assert int(kept_h[si]) == kept


@pytest.mark.parametrize("U", [300, 1200])
def test_select_scores_at_division_edges(U):
    """Unit scores floor(W_u / len_u) where the quotient sits just below, at and just above an
    integer, around 2^53 and far above it (both select paths), against the oracle."""
    from paper_2609_34653_amd import omnitide as ot
    rng = np.random.default_rng(U + 53)
    lens = rng.integers(1, 3000, size=U)
    first = np.concatenate([[0], np.cumsum(lens)[:-1]])
    last = first + lens - 1
    kind = rng.integers(0, 4, size=U)
    q = rng.integers(1, 1 << 40, size=U, dtype=np.int64)
    wsum = np.where(kind == 0, q * lens + rng.integers(-1, 2, size=U),          # near multiples
                    np.where(kind == 1, (1 << 53) + rng.integers(-3, 4, size=U),  # around 2^53
                             np.where(kind == 2, rng.integers(1 << 53,
                                                              np.maximum(lens << 50,
                                                                         (1 << 53) + 1),
                                                              dtype=np.int64),
                                      rng.integers(0, 1 << 53, size=U, dtype=np.int64))))
    wsum = np.maximum(wsum, 0).astype(np.int64)
    flags = np.zeros(U, np.int64)
    budget, recent = int(lens.sum() // 3), 2000
    i32 = lambda a: dev(np.asarray(a, np.int32))   # noqa: E731
    sc_d = torch.zeros(U, dtype=torch.int64, device="cuda")
    keep_d = torch.zeros(U, dtype=torch.uint8, device="cuda")
    kept_d = torch.zeros(1, dtype=torch.int32, device="cuda")
    stat = torch.zeros(1, dtype=torch.int32, device="cuda")
    ot.omnitide_select_units(dev(wsum), i32(lens), i32(first), i32(last), i32(flags), 1, U,
                             budget, recent, sc_d, keep_d, kept_d, stat)
    torch.cuda.synchronize()
    assert int(host(stat)[0]) == 0
    score, keep, kept = oracle.select_units(wsum, lens, first, last, flags, budget, recent)
    assert np.array_equal(host(sc_d), score)
    assert np.array_equal(host(keep_d), keep)
    assert int(host(kept_d)[0]) == kept


@pytest.mark.parametrize("U", [40, 600])
def test_select_score_out_of_key_range_reported(U):
    """A score of 2^51 or more does not fit the ranking key: E_RANGE, nothing kept (both
    kernel shapes); a broken unit structure in the same call reports E_TAGS first."""
    from paper_2609_34653_amd import omnitide as ot
    lens = np.full(U, 10)
    first = np.arange(U) * 10
    last = first + 9
    wsum = np.full(U, 1000, np.int64)
    wsum[7] = 10 << 51
    i32 = lambda a: dev(np.asarray(a, np.int32))   # noqa: E731
    for broken, code in ((False, ot.E_RANGE), (True, ot.E_TAGS)):
        lst = last.copy()
        if broken:
            lst[3] += 1
        sc_d = torch.zeros(U, dtype=torch.int64, device="cuda")
        keep_d = torch.ones(U, dtype=torch.uint8, device="cuda")
        kept_d = torch.ones(1, dtype=torch.int32, device="cuda")
        stat = torch.zeros(1, dtype=torch.int32, device="cuda")
        ot.omnitide_select_units(dev(wsum), i32(lens), i32(first), i32(lst), i32(np.zeros(U)), 1,
                                 U, 200, 30, sc_d, keep_d, kept_d, stat)
        torch.cuda.synchronize()
        assert int(host(stat)[0]) == code
        assert not host(keep_d).any() and int(host(kept_d)[0]) == 0
