"""Native (logical-only) layout on the GPU vs the CPU oracle, through the C ABI: attention over a
holey span.

Bar: attention within max |err| <= 1e-2 and mean |err| <= 1e-3 of the float64 oracle on the
same bf16 inputs (the prefill bar); full-size pools compare sampled query rows the oracle
computes one by one.
"""
import numpy as np
import pytest
import torch

import oracle
import streamgen as sg
from tests._util import storage_np
from tests.test_gpu_parity import dev, host

pytestmark = pytest.mark.gpu

MAX_ABS, MEAN_ABS = 1e-2, 1e-3


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_34653_amd import omnitide
    omnitide.lib()
    yield


def bf16(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(torch.bfloat16)


def run_span_attn(q, k, v, key_pos, span, q_pos0, scale, expect_status=0, skip=True):
    """q [n_seg, L, Hq, d], k/v [n_seg, cap, Hkv, d] bf16 (CPU); key_pos [n_seg, cap].
    skip: True (tile skipping), False (the full span) or "pos" (position order)."""
    from paper_2609_34653_amd import omnitide as ot
    n_seg, L, Hq, d = q.shape
    cap, Hkv = k.shape[1], k.shape[2]
    out = torch.full((n_seg, L, Hq, d), float("nan"), device="cuda")
    nb = ot.omnitide_span_attn_workspace_bytes(n_seg, cap, L, Hq, Hkv, d)
    ws = torch.zeros(nb, dtype=torch.uint8, device="cuda")
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    ot.omnitide_span_attn(q.cuda(), k.cuda(), v.cuda(),
                          dev(np.asarray(key_pos, np.int32).reshape(-1)),
                          dev(np.asarray(span, np.int32)), dev(np.asarray(q_pos0, np.int32)),
                          scale, out, ws, st, skip_empty_tiles=skip is True,
                          position_order=skip == "pos")
    torch.cuda.synchronize()
    assert int(host(st)[0]) == expect_status
    return host(out)


def check(out, q, k, v, key_pos, span, q_pos0, scale):
    """Every query row against the oracle; mean absolute error over the whole output.  out: one
    output or a list of outputs of the same call (one oracle evaluation for all)."""
    f = lambda t: oracle.to_f64(storage_np(t), "bf16")  # noqa: E731
    L = q.shape[0]
    # only occupied slots can be visible: hand the oracle those (in slot order)
    occ = np.nonzero(np.asarray(key_pos)[:span] >= 0)[0]
    k, v, key_pos, span = k[occ], v[occ], np.asarray(key_pos)[occ], len(occ)
    ref = oracle.span_attention(f(q), f(k), f(v), key_pos, span, q_pos0, scale)
    for o in (out if isinstance(out, (list, tuple)) else [out]):
        assert o.shape[0] == L
        err = np.abs(o.astype(np.float64) - ref)
        assert np.isfinite(o).all()
        assert err.max() <= MAX_ABS, err.max()
        assert err.mean() <= MEAN_ABS, err.mean()


def random_span_pool(rng, cap, L, Hkv, d, fill, empty_tiles=True, nan_holes=True):
    """Entries at random slots (some whole 64-slot tiles empty), dense positions in a random
    temporal order of runs, the chunk in the lowest free run of L slots."""
    occ = rng.random(cap - L) < fill
    if empty_tiles:
        for t in range(0, cap - L, 64):
            if rng.random() < 0.25:
                occ[t:t + 64] = False
    uid = np.full(cap, -1)
    uid[:cap - L][occ] = 0
    s0 = oracle.place_chunk(uid, L, cap)
    hist = np.nonzero(uid >= 0)[0]
    key_pos = np.full(cap, -1)
    key_pos[hist] = rng.permutation(len(hist))          # any physical order of positions
    key_pos[s0:s0 + L] = len(hist) + np.arange(L)
    span = int(np.nonzero(key_pos >= 0)[0][-1]) + 1
    k = rng.standard_normal((cap, Hkv, d)).astype(np.float32)
    v = rng.standard_normal((cap, Hkv, d)).astype(np.float32)
    if nan_holes:
        k[key_pos < 0] = np.nan
        v[key_pos < 0] = np.inf
    return bf16(k), bf16(v), key_pos, span, len(hist)


@pytest.mark.parametrize("cap,L,Hq,Hkv,d,fill,seed,skip", [
    (700, 37, 8, 2, 128, 0.5, 0, True),       # ragged span, several tiles, GQA 4
    (2000, 100, 4, 4, 64, 0.3, 1, True),      # no grouping, d = 64
    (1500, 200, 32, 8, 128, 0.9, 2, True),    # nearly full, chunk 200
    (5000, 64, 8, 1, 128, 0.1, 3, True),      # sparse: many empty tiles
    (5000, 64, 8, 1, 128, 0.1, 3, False),     # the same, every tile traversed
    (2000, 100, 4, 4, 64, 0.3, 1, False),
    (700, 37, 8, 2, 128, 0.5, 0, "pos"),      # position order: the same pools
    (2000, 100, 4, 4, 64, 0.3, 1, "pos"),
    (1500, 200, 32, 8, 128, 0.9, 2, "pos"),
    (5000, 64, 8, 1, 128, 0.1, 3, "pos"),
    (9000, 1, 8, 8, 64, 0.02, 4, "pos"),      # one query over a sparse pool
    (3000, 150, 16, 2, 128, 0.7, 5, "pos"),   # 8 query heads per KV head
])
def test_span_attention_random_pools(cap, L, Hq, Hkv, d, fill, seed, skip):
    rng = np.random.default_rng(seed)
    k, v, key_pos, span, q_pos0 = random_span_pool(rng, cap, L, Hkv, d, fill)
    q = bf16(rng.standard_normal((L, Hq, d)))
    scale = d ** -0.5
    out = run_span_attn(q[None], k[None], v[None], key_pos[None], [span], [q_pos0], scale,
                        skip=skip)
    check(out[0], q, k, v, key_pos, span, q_pos0, scale)


def test_span_attention_several_segments():
    rng = np.random.default_rng(5)
    cap, L, Hq, Hkv, d = 1200, 50, 8, 2, 128
    pools = [random_span_pool(rng, cap, L, Hkv, d, f) for f in (0.2, 0.6, 0.95)]
    q = bf16(rng.standard_normal((3, L, Hq, d)))
    args = (q, torch.stack([p[0] for p in pools]), torch.stack([p[1] for p in pools]),
            np.stack([p[2] for p in pools]), [p[3] for p in pools], [p[4] for p in pools], 0.1)
    out = run_span_attn(*args)
    out_p = run_span_attn(*args, skip="pos")
    for i, (k, v, kp, span, qp) in enumerate(pools):
        check([out[i], out_p[i]], q[i], k, v, kp, span, qp, 0.1)


def test_dense_positions_match_chunk_attention():
    """key_pos = slot index and q_pos0 = span - L: the contiguous chunk attention."""
    from paper_2609_34653_amd import omnitide as ot
    rng = np.random.default_rng(6)
    cap, L, Hq, Hkv, d, n = 3000, 300, 16, 4, 128, 2345
    k = bf16(rng.standard_normal((1, cap, Hkv, d)))
    v = bf16(rng.standard_normal((1, cap, Hkv, d)))
    q = bf16(rng.standard_normal((1, L, Hq, d)))
    kp = np.where(np.arange(cap) < n, np.arange(cap), -1)
    out = run_span_attn(q, k, v, kp[None], [n], [n - L], 0.09)
    ref = torch.zeros(1, L, Hq, d, device="cuda")
    nb = ot.omnitide_attn_workspace_bytes(1, cap, L, Hq, Hkv, d)
    ws = torch.zeros(max(nb, 1), dtype=torch.uint8, device="cuda")
    ot.omnitide_chunk_attn(q.cuda(), k.cuda(), v.cuda(), dev(np.array([n], np.int32)), 0.09, ref,
                           ws)
    torch.cuda.synchronize()
    assert np.abs(out - host(ref)).max() <= 2e-3
    check(out[0], q[0], k[0], v[0], kp, n, n - L, 0.09)


def chunk_attn_compacted(q, k, v, key_pos, n, scale):
    """omnitide_chunk_attn over the entries of a holey pool moved to slots 0 .. n-1 in position
    order (the same capacity, so the same split count)."""
    from paper_2609_34653_amd import omnitide as ot
    n_seg, cap, Hkv, d = k.shape
    L, Hq = q.shape[1], q.shape[2]
    kc, vc = torch.zeros_like(k), torch.zeros_like(v)
    for i in range(n_seg):
        slots = np.argsort(np.where(key_pos[i] >= 0, key_pos[i], np.iinfo(np.int64).max),
                           kind="stable")[:n[i]]
        assert np.array_equal(key_pos[i][slots], np.arange(n[i]))
        kc[i, :n[i]] = k[i, torch.from_numpy(slots)]
        vc[i, :n[i]] = v[i, torch.from_numpy(slots)]
    out = torch.zeros(n_seg, L, Hq, d, device="cuda")
    nb = ot.omnitide_attn_workspace_bytes(n_seg, cap, L, Hq, Hkv, d)
    ws = torch.zeros(max(nb, 1), dtype=torch.uint8, device="cuda")
    ot.omnitide_chunk_attn(q.cuda(), kc.cuda(), vc.cuda(), dev(np.asarray(n, np.int32)), scale,
                           out, ws)
    torch.cuda.synchronize()
    return host(out)


@pytest.mark.parametrize("cap,L,Hq,Hkv,d,fills,seed", [
    (3000, 300, 16, 4, 128, (0.4,), 7),
    (2500, 77, 8, 2, 64, (0.15, 0.8), 8),     # two segments, d = 64, ragged last tile
])
def test_position_order_bitwise_equals_compacted(cap, L, Hq, Hkv, d, fills, seed):
    """Position order visits the same tiles, in the same order, with the same masks as the chunk
    attention over the compacted pool: the outputs agree bit for bit."""
    rng = np.random.default_rng(seed)
    pools = [random_span_pool(rng, cap, L, Hkv, d, f, nan_holes=False) for f in fills]
    q = bf16(rng.standard_normal((len(fills), L, Hq, d)))
    k, v = torch.stack([p[0] for p in pools]), torch.stack([p[1] for p in pools])
    kp = np.stack([p[2] for p in pools])
    n = [p[4] + L for p in pools]
    out = run_span_attn(q, k, v, kp, [p[3] for p in pools], [p[4] for p in pools], 0.08,
                        skip="pos")
    ref = chunk_attn_compacted(q, k, v, kp, n, 0.08)
    assert np.array_equal(out, ref)


def test_position_order_errors_reported():
    """Entries that are not the positions 0 .. q_pos0 + L - 1 once each: OMNITIDE_E_TAGS on the
    device (a repeated, a missing or a too-large position, q_pos0 out of range); an invalid
    span: OMNITIDE_E_CAPACITY."""
    rng = np.random.default_rng(10)
    k, v, kp, span, qp = random_span_pool(rng, 1500, 60, 2, 128, 0.5, nan_holes=False)
    q = bf16(rng.standard_normal((1, 60, 8, 128)))
    hist = np.nonzero((kp >= 0) & (kp < qp))[0]
    run = lambda kp2, span2=span, qp2=qp, st=-17: run_span_attn(  # noqa: E731
        q, k[None], v[None], kp2[None], [span2], [qp2], 0.1, expect_status=st, skip="pos")
    run(kp, st=0)
    dup = kp.copy()
    dup[hist[3]] = kp[hist[10]]                 # position held twice (and one missing)
    run(dup)
    big = kp.copy()
    big[hist[5]] = qp + 60                      # position n
    run(big)
    gone = kp.copy()
    gone[hist[7]] = -1                          # one position missing
    run(gone)
    run(kp, qp2=-1)
    run(kp, qp2=span - 59)                      # q_pos0 + L > span
    run(kp, qp2=qp - 1)                         # the chunk's last position >= n
    run(kp, span2=1501, st=-5)


def test_position_order_workspace_reused_across_layouts():
    """The position index is built without clearing: one workspace (NaN-filled at first) serves
    calls over different layouts in turn, a malformed one among them, and each call sees only
    its own entries (stale index entries of earlier calls neither leak into the output nor
    raise a false OMNITIDE_E_TAGS)."""
    from paper_2609_34653_amd import omnitide as ot
    rng = np.random.default_rng(15)
    cap, L, Hq, Hkv, d = 2400, 48, 8, 2, 128
    pools = [random_span_pool(rng, cap, L, Hkv, d, f, nan_holes=False) for f in (0.3, 0.7, 0.5)]
    q = bf16(rng.standard_normal((1, L, Hq, d)))
    nb = ot.omnitide_span_attn_workspace_bytes(1, cap, L, Hq, Hkv, d)
    ws = torch.full((nb // 4 + 1,), float("nan"), device="cuda").view(torch.uint8)[:nb]
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    out = torch.zeros(1, L, Hq, d, device="cuda")

    def call(k, v, kp, span, qp, expect):
        st.zero_()
        ot.omnitide_span_attn(q.cuda(), k[None].cuda(), v[None].cuda(),
                              dev(np.asarray(kp, np.int32)), dev(np.array([span], np.int32)),
                              dev(np.array([qp], np.int32)), 0.1, out, ws, st,
                              position_order=True)
        torch.cuda.synchronize()
        assert int(host(st)[0]) == expect
        return host(out)[0]

    for k, v, kp, span, qp in pools:
        check(call(k, v, kp, span, qp, 0), q[0], k, v, kp, span, qp, 0.1)
    k, v, kp, span, qp = pools[1]
    gone = kp.copy()
    gone[np.nonzero((kp >= 0) & (kp < qp))[0][17]] = -1   # its slot_of entry is stale now
    call(k, v, gone, span, qp, -17)
    dup = kp.copy()
    a, b = np.nonzero((kp >= 0) & (kp < qp))[0][[5, 40]]
    dup[a] = kp[b]
    call(k, v, dup, span, qp, -17)
    check(call(k, v, kp, span, qp, 0), q[0], k, v, kp, span, qp, 0.1)


def native_80k(keep_whole=True):
    """The 80K history after the whole-unit plan, evicted in place, the chunk in the lowest run
    of empty slots."""
    cfg = sg.CONFIG_BY_NAME["history_80k"]
    stream = sg.make_stream(cfg)
    lay, seg = stream.layout, stream.segment(0)
    k = storage_np(seg.k_hist)
    sc = oracle.score_units(k, cfg.dtype, lay.unit_id, lay.modality, cfg.weights, lay.n_units)
    _, keep, kept = oracle.select_units(sc["wsum"], sc["len"], sc["first"], sc["last"],
                                        sc["flags"], cfg.budget, cfg.recent)
    ev = oracle.evict_logical(lay.unit_id, lay.pos, np.where(keep != 0, sc["len"], 0),
                              lay.n_units)
    L = lay.chunk_len
    cap = lay.n_slots + L
    uid = np.concatenate([ev["unit_id"], np.full(L, -1)])
    s0 = oracle.place_chunk(uid, L, cap)
    key_pos = np.concatenate([ev["pos"], np.full(L, -1)])
    key_pos[s0:s0 + L] = ev["kept"] + np.arange(L)
    kk = torch.cat([seg.k_hist, torch.zeros(L, *seg.k_hist.shape[1:], dtype=torch.bfloat16)])
    vv = torch.cat([seg.v_hist, torch.zeros(L, *seg.v_hist.shape[1:], dtype=torch.bfloat16)])
    kk[s0:s0 + L] = seg.k_chunk
    vv[s0:s0 + L] = seg.v_chunk
    span = int(np.nonzero(key_pos >= 0)[0][-1]) + 1
    return cfg, seg.q, kk, vv, key_pos, span, ev["kept"], s0


def test_span_attention_native_80k():
    cfg, q, k, v, key_pos, span, q_pos0, s0 = native_80k()
    assert s0 < span - 665 and span > 60000, "the chunk fills a hole, the span stays long"
    outs = [run_span_attn(q[None], k[None], v[None], key_pos[None], [span], [q_pos0], cfg.scale,
                          skip=skip)[0] for skip in (True, False, "pos")]
    check(outs, q, k, v, key_pos, span, q_pos0, cfg.scale)
    # position order over the native pool = the chunk attention over the compacted pool
    ref = chunk_attn_compacted(q[None], k[None], v[None], key_pos[None], [q_pos0 + 665],
                               cfg.scale)
    assert np.array_equal(outs[2], ref[0])


def test_span_attention_capacity_error():
    rng = np.random.default_rng(9)
    k, v, kp, span, qp = random_span_pool(rng, 500, 40, 2, 64, 0.5, nan_holes=False)
    q = bf16(rng.standard_normal((1, 40, 4, 64)))
    out = run_span_attn(q, k[None], v[None], kp[None], [501], [qp], 0.1,
                        expect_status=-5)
    assert np.all(np.isnan(out))
    out = run_span_attn(q, k[None], v[None], kp[None], [39], [qp], 0.1, expect_status=-5)
    assert np.all(np.isnan(out))


# ------------------------------------------------------------------------------ layout kernels

def i32(a):
    return dev(np.asarray(a, np.int32))


def place_ws(cap):
    from paper_2609_34653_amd import omnitide as ot
    return torch.zeros(ot.omnitide_place_chunk_workspace_bytes(1, cap), dtype=torch.uint8,
                       device="cuda")


def native_state(cfg_name, extra=None, plan="whole", seed_keep=None):
    """GPU pool of capacity n_slots + L (+extra) with the stream's tags, scored on the GPU, and
    the retention plan (whole-unit select, or arbitrary kept prefixes) on the host."""
    from paper_2609_34653_amd import omnitide as ot
    cfg = sg.CONFIG_BY_NAME[cfg_name]
    stream = sg.make_stream(cfg)
    lay, seg = stream.layout, stream.segment(0)
    L = lay.chunk_len
    cap = lay.n_slots + L + (extra or 0)
    pad = cap - lay.n_slots
    uid = np.concatenate([lay.unit_id, np.full(pad, -1)]).astype(np.int32)
    pos = np.concatenate([lay.pos, np.full(pad, -1)]).astype(np.int32)
    mod = np.concatenate([lay.modality, np.full(pad, 1)]).astype(np.uint8)
    kdt = seg.k_hist.dtype
    k = torch.cat([seg.k_hist, torch.zeros(pad, *seg.k_hist.shape[1:], dtype=kdt)])
    v = torch.cat([seg.v_hist, torch.zeros(pad, *seg.v_hist.shape[1:], dtype=kdt)])
    k[lay.n_slots:] = 3.0                               # recognisable bytes in the free tail
    k_np, v_np = storage_np(k), storage_np(v)
    sc = oracle.score_units(storage_np(seg.k_hist), cfg.dtype, lay.unit_id, lay.modality,
                            cfg.weights, lay.n_units)
    if plan == "whole":
        _, keep, _ = oracle.select_units(sc["wsum"], sc["len"], sc["first"], sc["last"],
                                         sc["flags"], cfg.budget, cfg.recent)
        keep_len = np.where(keep != 0, sc["len"], 0)
    else:
        rng = np.random.default_rng(seed_keep)
        keep_len = rng.integers(-2, sc["len"] + 3)
        keep_len[rng.random(lay.n_units) < 0.3] = 0
    g = dict(k=k.cuda()[None].contiguous(), v=v.cuda()[None].contiguous(), uid=i32(uid),
             pos=i32(pos), mod=dev(mod), len=i32(sc["len"]), keep_len=i32(keep_len),
             keep=dev((keep_len > 0).astype(np.uint8)),
             remap=i32(np.zeros(lay.n_units)), kept=i32([0]), nku=i32([0]), span=i32([0]),
             ws=torch.zeros(ot.omnitide_evict_native_workspace_bytes(1, lay.n_units),
                            dtype=torch.uint8, device="cuda"),
             st=i32([0]))
    h = dict(uid=uid, pos=pos, mod=mod, k=k_np, v=v_np, keep_len=keep_len, sc=sc)
    return cfg, lay, seg, g, h


def gpu_evict(lay, g, use_len=True):
    from paper_2609_34653_amd import omnitide as ot
    ot.omnitide_evict_native(g["uid"], g["pos"], 1, lay.n_units, g["len"], g["remap"], g["kept"],
                             g["nku"], g["span"], g["ws"],
                             keep=None if use_len else g["keep"],
                             keep_len=g["keep_len"] if use_len else None, d_status=g["st"])
    torch.cuda.synchronize()


def check_evict(lay, g, h):
    kl = np.minimum(np.maximum(h["keep_len"], 0), h["sc"]["len"])
    ev = oracle.evict_logical(h["uid"], h["pos"], kl, lay.n_units)
    assert int(host(g["st"])[0]) == 0
    assert np.array_equal(host(g["uid"]), ev["unit_id"])
    assert np.array_equal(host(g["pos"]), ev["pos"])
    assert np.array_equal(host(g["remap"]), ev["unit_remap"])
    assert int(host(g["kept"])[0]) == ev["kept"]
    assert int(host(g["nku"])[0]) == ev["n_kept_units"]
    assert int(host(g["span"])[0]) == oracle.span_of(ev["unit_id"])
    return ev


@pytest.mark.parametrize("cfg_name,plan", [("tiny_1p6k_f32", "whole"),
                                           ("single_layer_8k", "prefix"),
                                           ("history_80k", "whole"), ("history_80k", "prefix")])
def test_evict_native_parity(cfg_name, plan):
    cfg, lay, seg, g, h = native_state(cfg_name, plan=plan, seed_keep=3)
    gpu_evict(lay, g, use_len=plan == "prefix")
    check_evict(lay, g, h)
    # K/V are not touched by logical eviction
    assert np.array_equal(storage_np(g["k"][0]), h["k"])


def test_evict_native_tag_error():
    cfg, lay, seg, g, h = native_state("single_layer_8k")
    bad = h["pos"].copy()
    s = int(np.nonzero(h["uid"] == 3)[0][0])
    bad[s] = bad[s] + 10_000                             # outside unit 3's positions
    g["pos"] = i32(bad)
    gpu_evict(lay, g)
    assert int(host(g["st"])[0]) == -17


@pytest.mark.parametrize("cfg_name,P,T", [("single_layer_8k", 64, 1), ("single_layer_8k", 64, 8),
                                          ("history_80k", 256, 1), ("history_80k", 256, 40),
                                          ("history_80k", 256, 10_000)])
def test_pack_suffix_parity(cfg_name, P, T):
    from paper_2609_34653_amd import omnitide as ot
    cfg, lay, seg, g, h = native_state(cfg_name, plan="whole")
    gpu_evict(lay, g)
    ev = check_evict(lay, g, h)
    cap = len(h["uid"])
    H, d = seg.k_hist.shape[1], seg.k_hist.shape[2]
    nb = ot.omnitide_pack_suffix_workspace_bytes(0 if cfg.dtype == "bf16" else 1, 1, cap, H, d)
    ws = torch.zeros(nb, dtype=torch.uint8, device="cuda")
    cut, moved = i32([7]), i32([7])
    ot.omnitide_pack_suffix(g["k"], g["v"], P, T, g["uid"], g["mod"], g["pos"], g["span"], cut,
                            moved, ws)
    torch.cuda.synchronize()
    c, ns = oracle.plan_suffix(ev["unit_id"] >= 0, P, T)
    assert int(host(cut)[0]) == c
    assert int(host(g["span"])[0]) == ns
    if c < 0:
        assert int(host(moved)[0]) == 0
        assert np.array_equal(host(g["uid"]), ev["unit_id"])
        return
    pk = oracle.pack_suffix(h["k"], h["v"], ev["unit_id"], h["mod"], ev["pos"], c)
    assert int(host(moved)[0]) == pk["moved"] and pk["moved"] > 0
    assert np.array_equal(host(g["uid"]), pk["unit_id"])
    assert np.array_equal(host(g["pos"]), pk["pos"])
    assert np.array_equal(host(g["mod"]), pk["modality"])
    assert np.array_equal(storage_np(g["k"][0]), pk["k"])
    assert np.array_equal(storage_np(g["v"][0]), pk["v"])


def test_place_chunk_parity_and_native_attention():
    """80K history: eviction, the chunk into the lowest empty run, attention over the span."""
    from paper_2609_34653_amd import omnitide as ot
    cfg, lay, seg, g, h = native_state("history_80k")
    gpu_evict(lay, g)
    ev = check_evict(lay, g, h)
    L = lay.chunk_len
    cap = len(h["uid"])
    slot = i32([-9])
    ot.omnitide_place_chunk(g["k"], g["v"], g["uid"], g["mod"], g["pos"],
                            seg.k_chunk.cuda()[None].contiguous(),
                            seg.v_chunk.cuda()[None].contiguous(), dev(lay.chunk_modality),
                            dev(lay.chunk_unit), g["kept"], g["nku"], slot, g["span"],
                            place_ws(cap), d_status=g["st"])
    torch.cuda.synchronize()
    assert int(host(g["st"])[0]) == 0
    s0 = oracle.place_chunk(ev["unit_id"], L, cap)
    assert int(host(slot)[0]) == s0
    uid = ev["unit_id"].copy()
    pos = ev["pos"].copy()
    uid[s0:s0 + L] = ev["n_kept_units"] + lay.chunk_unit
    pos[s0:s0 + L] = ev["kept"] + np.arange(L)
    assert np.array_equal(host(g["uid"]), uid) and np.array_equal(host(g["pos"]), pos)
    assert np.array_equal(host(g["mod"])[s0:s0 + L], lay.chunk_modality)
    kk = h["k"].copy()
    kk[s0:s0 + L] = storage_np(seg.k_chunk)
    assert np.array_equal(storage_np(g["k"][0]), kk)
    span = int(host(g["span"])[0])
    assert span == oracle.span_of(uid)
    # attention over the span with the device-built layout
    nb = ot.omnitide_span_attn_workspace_bytes(1, cap, L, cfg.n_q_heads, cfg.n_kv_heads,
                                               cfg.head_dim)
    ws = torch.zeros(nb, dtype=torch.uint8, device="cuda")
    out = torch.zeros(1, L, cfg.n_q_heads, cfg.head_dim, device="cuda")
    ot.omnitide_span_attn(seg.q.cuda()[None].contiguous(), g["k"], g["v"], g["pos"], g["span"],
                          g["kept"], cfg.scale, out, ws, g["st"])
    torch.cuda.synchronize()
    assert int(host(g["st"])[0]) == 0
    kt, vt = torch.from_numpy(kk.view(np.int16)).view(torch.bfloat16), g["v"][0].cpu()
    check(host(out)[0], seg.q, kt, vt, pos, span, ev["kept"], cfg.scale)


def test_place_chunk_capacity_error():
    from paper_2609_34653_amd import omnitide as ot
    cfg, lay, seg, g, h = native_state("single_layer_8k")
    # nothing evicted and no free tail: the pool is full
    uid = np.where(h["uid"] >= 0, h["uid"], 0).astype(np.int32)
    g["uid"] = i32(uid)
    slot = i32([5])
    span = i32([5])
    ot.omnitide_place_chunk(g["k"], g["v"], g["uid"], g["mod"], g["pos"],
                            seg.k_chunk.cuda()[None].contiguous(),
                            seg.v_chunk.cuda()[None].contiguous(), dev(lay.chunk_modality),
                            dev(lay.chunk_unit), g["kept"], g["nku"], slot, span,
                            place_ws(len(uid)), d_status=g["st"])
    torch.cuda.synchronize()
    assert int(host(g["st"])[0]) == -5 and int(host(slot)[0]) == -1
    assert np.array_equal(host(g["uid"]), uid)


def test_native_kernels_several_segments():
    """Eviction, suffix packing and placement on two segments in one call each (segment 0: the
    whole-unit plan, segment 1: arbitrary kept prefixes)."""
    from paper_2609_34653_amd import omnitide as ot
    cfg, lay, seg, g0, h0 = native_state("single_layer_8k", plan="whole")
    _, _, _, g1, h1 = native_state("single_layer_8k", plan="prefix", seed_keep=9)
    U, cap, L = lay.n_units, len(h0["uid"]), lay.chunk_len
    cat = lambda key: torch.cat([g0[key].view(-1), g1[key].view(-1)]).contiguous()  # noqa: E731
    uid, pos, mod = cat("uid"), cat("pos"), cat("mod")
    k = torch.cat([g0["k"], g1["k"]]).contiguous()
    v = torch.cat([g0["v"], g1["v"]]).contiguous()
    remap = i32(np.zeros(2 * U))
    kept, nku, span, st = i32([0, 0]), i32([0, 0]), i32([0, 0]), i32([0])
    ws = torch.zeros(ot.omnitide_evict_native_workspace_bytes(2, U), dtype=torch.uint8,
                     device="cuda")
    ot.omnitide_evict_native(uid, pos, 2, U, cat("len"), remap, kept, nku, span, ws,
                             keep_len=cat("keep_len"), d_status=st)
    H, d = seg.k_hist.shape[1], seg.k_hist.shape[2]
    wsp = torch.zeros(ot.omnitide_pack_suffix_workspace_bytes(0, 2, cap, H, d),
                      dtype=torch.uint8, device="cuda")
    cut, moved = i32([0, 0]), i32([0, 0])
    ot.omnitide_pack_suffix(k, v, 64, 1, uid, mod, pos, span, cut, moved, wsp)
    kc = torch.stack([seg.k_chunk, seg.k_chunk]).cuda().contiguous()
    vc = torch.stack([seg.v_chunk, seg.v_chunk]).cuda().contiguous()
    slot = i32([0, 0])
    wsc = torch.zeros(ot.omnitide_place_chunk_workspace_bytes(2, cap), dtype=torch.uint8,
                      device="cuda")
    ot.omnitide_place_chunk(k, v, uid, mod, pos, kc, vc, dev(lay.chunk_modality),
                            dev(lay.chunk_unit), kept, nku, slot, span, wsc, d_status=st)
    torch.cuda.synchronize()
    assert int(host(st)[0]) == 0
    for si, h in enumerate((h0, h1)):
        kl = np.minimum(np.maximum(h["keep_len"], 0), h["sc"]["len"])
        ev = oracle.evict_logical(h["uid"], h["pos"], kl, U)
        assert np.array_equal(host(remap)[si * U:(si + 1) * U], ev["unit_remap"])
        assert int(host(kept)[si]) == ev["kept"] and int(host(nku)[si]) == ev["n_kept_units"]
        c, _ = oracle.plan_suffix(ev["unit_id"] >= 0, 64, 1)
        assert int(host(cut)[si]) == c
        if c >= 0:
            pk = oracle.pack_suffix(h["k"], h["v"], ev["unit_id"], h["mod"], ev["pos"], c)
        else:
            pk = dict(k=h["k"], v=h["v"], unit_id=ev["unit_id"], modality=h["mod"],
                      pos=ev["pos"], moved=0)
        assert int(host(moved)[si]) == pk["moved"]
        s0 = oracle.place_chunk(pk["unit_id"], L, cap)
        assert int(host(slot)[si]) == s0
        want_uid = pk["unit_id"].copy()
        want_pos = pk["pos"].copy()
        want_uid[s0:s0 + L] = ev["n_kept_units"] + lay.chunk_unit
        want_pos[s0:s0 + L] = ev["kept"] + np.arange(L)
        sl = slice(si * cap, (si + 1) * cap)
        assert np.array_equal(host(uid)[sl], want_uid)
        assert np.array_equal(host(pos)[sl], want_pos)
        want_k = pk["k"].copy()
        want_k[s0:s0 + L] = storage_np(seg.k_chunk)
        assert np.array_equal(storage_np(k[si]), want_k)
        assert int(host(span)[si]) == oracle.span_of(want_uid)


@pytest.mark.parametrize("cfg_name,plan,rope", [
    ("history_80k", "whole", (1.0e6, 128, 0)),          # the benchmark's rotary setting
    ("single_layer_8k", "prefix", (10000.0, 64, 0)),    # arbitrary kept prefixes, partial width
    ("tiny_1p6k_f32", "prefix", (10000.0, 32, 1)),      # float32 keys, interleaved pairs
])
def test_evict_native_rope_parity(cfg_name, plan, rope):
    """Eviction with the rotary adjustment: tags bit-exact, the keys of kept slots whose position
    shifts re-rotated in place within the rotary bound (half a storage ulp plus 2^-21 of the
    pair's length), every other key byte and all of V unchanged."""
    from paper_2609_34653_amd import omnitide as ot
    from tests.test_gpu_rope import pair_norm, ulp
    cfg, lay, seg, g, h = native_state(cfg_name, plan=plan, seed_keep=31)
    cap = len(h["uid"])
    style = ("half", "interleaved")[rope[2]]
    ws = torch.zeros(ot.omnitide_evict_native_rope_workspace_bytes(1, lay.n_units, cap),
                     dtype=torch.uint8, device="cuda")
    ot.omnitide_evict_native_rope(g["uid"], g["pos"], g["k"], 1, lay.n_units, g["len"],
                                  g["remap"], g["kept"], g["nku"], g["span"], ws, rope[0],
                                  rope[1], rope[2], keep_len=g["keep_len"], d_status=g["st"])
    torch.cuda.synchronize()
    assert int(host(g["st"])[0]) == 0
    kl = np.minimum(np.maximum(h["keep_len"], 0), h["sc"]["len"])
    ev = oracle.evict_logical(h["uid"], h["pos"], kl, lay.n_units, k=h["k"],
                              rope=dict(base=rope[0], dims=rope[1], style=style, dtype=cfg.dtype))
    assert np.array_equal(host(g["uid"]), ev["unit_id"])
    assert np.array_equal(host(g["pos"]), ev["pos"])
    assert int(host(g["kept"])[0]) == ev["kept"]
    kd = storage_np(g["k"][0])
    moved = (ev["unit_id"] >= 0) & (ev["pos"] != h["pos"])
    assert moved.sum() > 1000 or cfg_name == "tiny_1p6k_f32" and moved.sum() > 100
    assert np.array_equal(kd[~moved], h["k"][~moved])             # untouched rows: same bytes
    assert np.array_equal(storage_np(g["v"][0]), h["v"])           # values carry no position
    R = rope[1]
    assert np.array_equal(kd[moved][..., R:], h["k"][moved][..., R:])
    got = oracle.to_f64(kd[moved], cfg.dtype)[..., :R]
    want = ev["k_f64"][moved][..., :R]
    src = oracle.to_f64(h["k"][moved], cfg.dtype)
    bound = 0.5 * ulp(want, cfg.dtype) + 2.0 ** -21 * pair_norm(src, R, style)[..., :R]
    assert np.all(np.abs(got - want) <= bound)


def test_evict_native_rope_then_span_attention_equals_compaction():
    """On the 80K history: eviction with the rotary adjustment followed by attention over the
    span gives what rotary compaction followed by chunk attention gives (same keys at the same
    logical positions)."""
    from paper_2609_34653_amd import omnitide as ot
    from tests.test_gpu_parity import make_step, gpu_inputs
    cfg, lay, seg, g, h = native_state("history_80k")
    cap = len(h["uid"])
    L = lay.chunk_len
    rope = (1.0e6, 128, 0)
    ws = torch.zeros(ot.omnitide_evict_native_rope_workspace_bytes(1, lay.n_units, cap),
                     dtype=torch.uint8, device="cuda")
    ot.omnitide_evict_native_rope(g["uid"], g["pos"], g["k"], 1, lay.n_units, g["len"],
                                  g["remap"], g["kept"], g["nku"], g["span"], ws, *rope,
                                  keep=g["keep"], d_status=g["st"])
    ot.omnitide_place_chunk(g["k"], g["v"], g["uid"], g["mod"], g["pos"],
                            seg.k_chunk.cuda()[None].contiguous(),
                            seg.v_chunk.cuda()[None].contiguous(), dev(lay.chunk_modality),
                            dev(lay.chunk_unit), g["kept"], g["nku"], i32([0]), g["span"],
                            place_ws(cap), d_status=g["st"])
    nb = ot.omnitide_span_attn_workspace_bytes(1, cap, L, cfg.n_q_heads, cfg.n_kv_heads,
                                               cfg.head_dim)
    out_n = torch.zeros(1, L, cfg.n_q_heads, cfg.head_dim, device="cuda")
    ot.omnitide_span_attn(seg.q.cuda()[None].contiguous(), g["k"], g["v"], g["pos"], g["span"],
                          g["kept"], cfg.scale, out_n,
                          torch.zeros(nb, dtype=torch.uint8, device="cuda"), g["st"])
    st = make_step(cfg, lay)
    inp = gpu_inputs(lay, [seg])
    st.score(inp["k_hist"], inp["unit_id"], inp["modality"])
    st.select()
    st.compact(inp["k_hist"], inp["v_hist"], inp["unit_id"], inp["modality"], inp["pos"],
               inp["k_chunk"], inp["v_chunk"], inp["chunk_modality"], inp["chunk_unit"],
               rope=rope)
    st.attend(inp["q"], cfg.scale)
    torch.cuda.synchronize()
    assert int(host(g["st"])[0]) == 0 and int(host(st.d_status)[0]) == 0
    assert np.abs(host(out_n) - host(st.out)).max() <= 2e-3


def test_stream_loop_native_layouts_chained():
    """The stream loop's native and ordered-suffix (11 pages of 64 slots) layouts chained on the
    device for 24 steps, each step applying the whole-unit selection of the eager step (the
    unit ids of all layouts coincide).  Against the oracle chained on its own outputs (its own
    score and select of its own eager chain): eviction, suffix packing and chunk placement
    bit-exact at every step (every tag row, the chunk slot, the span, the kept count), the K/V
    bytes of every occupied slot, span attention (tile skipping and position order) on every
    query row, and the decode of the chunk's last token (all three traversals) after steps 12
    and 24."""
    from paper_2609_34653_amd import omnitide as ot
    from paper_2609_34653_amd.step import StreamStep
    cfg = sg.CONFIG_BY_NAME["stream_loop_64x665"]
    stream = sg.make_stream(cfg)
    lay, seg0 = stream.layout, stream.segment(0)
    U, L, page, steps = 512, lay.chunk_len, 64, 24
    H, d, Hq = cfg.n_kv_heads, cfg.head_dim, cfg.n_q_heads
    cap_e, cap_n = cfg.budget + L, 65536
    i32 = dict(dtype=torch.int32, device="cuda")
    pad = cap_n - lay.n_slots
    # eager chains: the device's drives the device layouts, the oracle's the oracle layouts
    src = dict(k=seg0.k_hist.cuda()[None], v=seg0.v_hist.cuda()[None], uid=dev(lay.unit_id),
               mod=dev(lay.modality), pos=dev(lay.pos))
    e_k, e_v = storage_np(seg0.k_hist), storage_np(seg0.v_hist)
    e_uid, e_mod, e_pos = lay.unit_id.astype(np.int64), lay.modality, lay.pos
    k0 = np.zeros((cap_n,) + e_k.shape[1:], e_k.dtype)
    k0[:lay.n_slots] = e_k
    v0 = np.zeros_like(k0)
    v0[:lay.n_slots] = e_v
    tags0 = (np.concatenate([lay.unit_id, np.full(pad, -1)]).astype(np.int64),
             np.concatenate([lay.modality, np.full(pad, 1)]).astype(np.uint8),
             np.concatenate([lay.pos, np.full(pad, -1)]).astype(np.int64))
    layouts = {}
    for name, T in (("native", 0), ("ordered_suffix", 11)):
        kd = torch.from_numpy(k0.view(np.int16)).view(torch.bfloat16).cuda()[None].contiguous()
        vd = torch.from_numpy(v0.view(np.int16)).view(torch.bfloat16).cuda()[None].contiguous()
        layouts[name] = dict(
            T=T, k=kd, v=vd, uid=dev(tags0[0].astype(np.int32)), mod=dev(tags0[1]),
            pos=dev(tags0[2].astype(np.int32)), remap=torch.zeros(U, **i32),
            kept=torch.zeros(1, **i32), nku=torch.zeros(1, **i32), span=torch.zeros(1, **i32),
            slot=torch.zeros(1, **i32), cut=torch.zeros(1, **i32), moved=torch.zeros(1, **i32),
            out=torch.zeros(1, L, Hq, d, device="cuda"),
            out_p=torch.zeros(1, L, Hq, d, device="cuda"),
            dec=torch.zeros(3, 1, Hq, d, device="cuda"), qpos=torch.zeros(1, **i32),
            o=dict(k=k0.copy(), v=v0.copy(), uid=tags0[0].copy(), mod=tags0[1].copy(),
                   pos=tags0[2].copy()))
    ws_e = torch.zeros(ot.omnitide_evict_native_workspace_bytes(1, U), dtype=torch.uint8,
                       device="cuda")
    ws_p = torch.zeros(ot.omnitide_pack_suffix_workspace_bytes(0, 1, cap_n, H, d),
                       dtype=torch.uint8, device="cuda")
    ws_c = torch.zeros(ot.omnitide_place_chunk_workspace_bytes(1, cap_n), dtype=torch.uint8,
                       device="cuda")
    ws_a = torch.zeros(ot.omnitide_span_attn_workspace_bytes(1, cap_n, L, Hq, H, d),
                       dtype=torch.uint8, device="cuda")
    ws_d = torch.zeros(ot.omnitide_decode_span_workspace_bytes(1, cap_n, 1, Hq, H, d),
                       dtype=torch.uint8, device="cuda")
    for t in range(steps):
        clay, cseg = sg.loop_chunk(cfg, t)
        ck, cv = storage_np(cseg.k_chunk), storage_np(cseg.v_chunk)
        st = StreamStep(n_seg=1, n_slots=src["k"].shape[1], n_units=U, n_q_heads=Hq,
                        n_kv_heads=H, head_dim=d, chunk_len=L, budget=cfg.budget,
                        recent=cfg.recent, page_size=cfg.page_size, weights=cfg.weights,
                        cap_dst=cap_e)
        st.score(src["k"], src["uid"], src["mod"])
        st.select()
        kc, vc = cseg.k_chunk.cuda()[None], cseg.v_chunk.cuda()[None]
        cm, cu = dev(clay.chunk_modality), dev(clay.chunk_unit)
        st.compact(src["k"], src["v"], src["uid"], src["mod"], src["pos"], kc, vc, cm, cu)
        check_now = t in (11, 23)
        for pl in layouts.values():
            ot.omnitide_evict_native(pl["uid"], pl["pos"], 1, U, st.unit_len, pl["remap"],
                                     pl["kept"], pl["nku"], pl["span"], ws_e, keep=st.keep,
                                     d_status=st.d_status)
            if pl["T"] > 0:
                ot.omnitide_pack_suffix(pl["k"], pl["v"], page, pl["T"], pl["uid"], pl["mod"],
                                        pl["pos"], pl["span"], pl["cut"], pl["moved"], ws_p)
            ot.omnitide_place_chunk(pl["k"], pl["v"], pl["uid"], pl["mod"], pl["pos"], kc, vc,
                                    cm, cu, pl["kept"], pl["nku"], pl["slot"], pl["span"], ws_c,
                                    d_status=st.d_status)
            if check_now:
                for key, po in (("out", False), ("out_p", True)):
                    ot.omnitide_span_attn(cseg.q.cuda()[None], pl["k"], pl["v"], pl["pos"],
                                          pl["span"], pl["kept"], cfg.scale, pl[key], ws_a,
                                          st.d_status, skip_empty_tiles=True,
                                          position_order=po)
                # the chunk's last token decodes: every tile, non-empty tiles, position order
                torch.add(pl["kept"], L - 1, out=pl["qpos"])
                qd = cseg.q.cuda()[None, L - 1:L].contiguous()
                for i, (sk, po) in enumerate(((False, False), (True, False), (True, True))):
                    ot.omnitide_decode_span_attn(qd, pl["k"], pl["v"], pl["pos"], pl["span"],
                                                 pl["qpos"], cfg.scale, pl["dec"][i], ws_d,
                                                 st.d_status, skip_empty_tiles=sk,
                                                 position_order=po)
        torch.cuda.synchronize()
        assert int(host(st.d_status)[0]) == 0, t
        # the oracle: its eager step gives the plan
        sc = oracle.score_units(e_k, "bf16", e_uid, e_mod, cfg.weights, U)
        _, keep, _ = oracle.select_units(sc["wsum"], sc["len"], sc["first"], sc["last"],
                                         sc["flags"], cfg.budget, cfg.recent)
        keep_len = np.where(keep != 0, sc["len"], 0)
        for name, pl in layouts.items():
            o = pl["o"]
            ev = oracle.evict_logical(o["uid"], o["pos"], keep_len, U)
            o["uid"], o["pos"] = ev["unit_id"], ev["pos"]
            if pl["T"] > 0:
                c, _ = oracle.plan_suffix(o["uid"] >= 0, page, pl["T"])
                assert int(host(pl["cut"])[0]) == c, (name, t)
                if c >= 0:
                    pk = oracle.pack_suffix(o["k"], o["v"], o["uid"], o["mod"], o["pos"], c)
                    o.update(k=pk["k"], v=pk["v"], uid=pk["unit_id"], mod=pk["modality"],
                             pos=pk["pos"])
            s0 = oracle.place_chunk(o["uid"], L, cap_n)
            o["k"][s0:s0 + L], o["v"][s0:s0 + L] = ck, cv
            o["uid"][s0:s0 + L] = ev["n_kept_units"] + clay.chunk_unit
            o["mod"][s0:s0 + L] = clay.chunk_modality
            o["pos"][s0:s0 + L] = ev["kept"] + np.arange(L)
            assert int(host(pl["slot"])[0]) == s0, (name, t)
            assert int(host(pl["kept"])[0]) == ev["kept"], (name, t)
            assert int(host(pl["span"])[0]) == oracle.span_of(o["uid"]), (name, t)
            uid_d, pos_d = host(pl["uid"]).astype(np.int64), host(pl["pos"]).astype(np.int64)
            assert np.array_equal(uid_d, o["uid"]), (name, t)
            assert np.array_equal(pos_d, o["pos"]), (name, t)
            occ = o["uid"] >= 0
            assert np.array_equal(host(pl["mod"])[occ], o["mod"][occ]), (name, t)
            if check_now:
                assert np.array_equal(storage_np(pl["k"][0])[occ], o["k"][occ]), (name, t)
                assert np.array_equal(storage_np(pl["v"][0])[occ], o["v"][occ]), (name, t)
                span = oracle.span_of(o["uid"])
                check([host(pl["out"])[0], host(pl["out_p"])[0]], cseg.q, bf16_view(o["k"]),
                      bf16_view(o["v"]), o["pos"], span, ev["kept"], cfg.scale)
                dec = host(pl["dec"])
                check_decode(dec, cseg.q[L - 1:L], o, span, ev["kept"] + L - 1, cfg.scale)
        # next eager state, on both sides
        cp = oracle.compact_kv(e_k, e_v, e_uid, e_mod, e_pos, keep, U, ck, cv,
                               clay.chunk_modality, clay.chunk_unit, cap_e, cfg.page_size)
        n = cp["n_ctx"]
        tail = cap_e - n
        e_k = np.concatenate([cp["k"], np.zeros((tail,) + cp["k"].shape[1:], cp["k"].dtype)])
        e_v = np.concatenate([cp["v"], np.zeros((tail,) + cp["v"].shape[1:], cp["v"].dtype)])
        e_uid = np.concatenate([cp["unit_id"], np.full(tail, -1)])
        e_mod = np.concatenate([cp["modality"], np.zeros(tail, np.int64)]).astype(np.uint8)
        e_pos = np.concatenate([cp["pos"], np.full(tail, -1)])
        src = dict(k=st.k_dst, v=st.v_dst, uid=st.unit_id_dst, mod=st.modality_dst,
                   pos=st.pos_dst)


def check_decode(outs, qd, o, span, q_pos0, scale):
    """Decode outputs [n, 1, Hq, d] of one token against the oracle over the occupied slots, to
    the decode bar (max 2e-5, mean 2e-6)."""
    f = lambda t: oracle.to_f64(storage_np(t), "bf16")  # noqa: E731
    occ = np.nonzero(o["pos"][:span] >= 0)[0]
    ref = oracle.span_attention(f(qd), f(bf16_view(o["k"][occ])), f(bf16_view(o["v"][occ])),
                                o["pos"][occ], len(occ), q_pos0, scale)
    for out in outs:
        err = np.abs(out.astype(np.float64) - ref)
        assert np.isfinite(out).all()
        assert err.max() <= 2e-5, err.max()
        assert err.mean() <= 2e-6, err.mean()


def bf16_view(a):
    """Storage values (uint16 bf16 bit patterns) as a CPU bf16 tensor."""
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)
