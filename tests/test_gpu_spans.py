"""HIP span plan and span compaction vs the CPU oracle, through the C ABI.

Bar: keep_len, keep_slot, kept_tokens and every compaction output bit-exact (integers and raw
KV bytes);
with rotary re-encoding, the rotated key elements within the bound of the rotary compaction
tests (half a storage ulp plus 2^-21 of the pair's length).
"""
import numpy as np
import pytest
import torch

import oracle
import streamgen as sg
from tests._util import storage_np
from tests.test_gpu_parity import dev, gpu_inputs, host, make_step
from tests.test_gpu_rope import pair_norm, ulp

pytestmark = pytest.mark.gpu

SYS, VIDEO, AUDIO, TEXT, MARK = 0, 1, 2, 3, 4


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_34653_amd import omnitide
    omnitide.lib()
    yield


def i32(a):
    return dev(np.asarray(a, np.int32))


def gpu_plan(length, first, last, flags, unit_id, modality, n_slots, params, n_seg=1):
    """Run omnitide_plan_spans on host arrays laid out [n_seg][U] and [n_seg][n_slots]; returns
    (keep_len, keep_slot, kept, status)."""
    from paper_2609_34653_amd import omnitide as ot
    U = len(length) // n_seg
    kl = torch.full((n_seg * U,), -7, dtype=torch.int32, device="cuda")
    ks = torch.full((n_seg * n_slots,), 7, dtype=torch.uint8, device="cuda")
    kt = torch.full((n_seg,), -7, dtype=torch.int32, device="cuda")
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = torch.full((max(1, ot.omnitide_plan_spans_workspace_bytes(n_seg, n_slots, U)),), 0xA5,
                    dtype=torch.uint8, device="cuda")
    ot.omnitide_plan_spans(i32(length), i32(first), i32(last), i32(flags), i32(unit_id),
                           dev(np.asarray(modality, np.uint8)), n_seg, n_slots, U,
                           params["low"], params["high"], params["recent"], params["sv"],
                           params["sa"], params["tb"], kl, ks, kt, ws, st)
    torch.cuda.synchronize()
    return host(kl), host(ks), host(kt), int(host(st)[0])


def oracle_plan(sc, modality, p):
    return oracle.plan_spans(modality, sc["len"], sc["first"], sc["last"], sc["flags"], p["low"],
                             p["high"], p["recent"], p["sv"], p["sa"], p["tb"])


def random_layout(rng, U, hole_p=0.2, mixed=True):
    """Contiguous unit runs in id order with empty slots between some of them; mixed units
    (grammar units, free tag sequences) or units of one modality."""
    units = (sg.random_mixed_units(rng, U, hi=40) if mixed else sg.random_units(rng, U, 1, 40))
    sys_u = rng.random(U) < 0.03
    unit_id, modality = [], []
    length = np.zeros(U, np.int64)
    for u in range(U):
        codes = sg.unit_codes(units[u]).astype(np.int64)
        if sys_u[u]:
            codes[int(rng.integers(len(codes)))] = SYS
        if rng.random() < 0.05:
            codes = codes[:0]                            # some units without slots
        if rng.random() < hole_p:
            gap = int(rng.integers(1, 5))
            unit_id += [-1] * gap
            modality += [int(rng.integers(0, 5))] * gap
        unit_id += [u] * len(codes)
        modality += codes.tolist()
        length[u] = len(codes)
    unit_id = np.array(unit_id, np.int64)
    modality = np.array(modality, np.int64)
    n = len(unit_id)
    first = np.full(U, n, np.int64)
    last = np.full(U, -1, np.int64)
    for s in range(n):
        u = unit_id[s]
        if u >= 0:
            first[u] = min(first[u], s)
            last[u] = s
    flags = np.zeros(U, np.int64)
    for u in range(U):
        if length[u] and np.any(modality[unit_id == u] == SYS):
            flags[u] = 1
    return dict(len=length, first=first, last=last, flags=flags, unit_id=unit_id), modality


def random_params(rng, total):
    high = int(rng.integers(0, total + 10))
    return dict(high=high, low=int(rng.integers(0, high + 1)),
                recent=int(rng.integers(0, max(total // 3, 1))), sv=int(rng.integers(0, 20)),
                sa=int(rng.integers(0, 8)), tb=int(rng.integers(0, 80)))


@pytest.mark.parametrize("U,seed", [(1, 0), (2, 1), (7, 2), (60, 3), (512, 4), (513, 5),
                                    (3000, 6), (8192, 7)])
@pytest.mark.parametrize("mixed", [True, False])
def test_plan_parity_random(U, seed, mixed):
    rng = np.random.default_rng(seed + (100 if mixed else 0))
    for trial in range(6):
        sc, modality = random_layout(rng, U, mixed=mixed)
        p = random_params(rng, int(sc["len"].sum()))
        if trial == 0:
            p["high"] = int(sc["len"].sum())             # nothing to trim
            p["low"] = min(p["low"], p["high"])
        want, wmask, wkept = oracle_plan(sc, modality, p)
        got, mask, kept, status = gpu_plan(sc["len"], sc["first"], sc["last"], sc["flags"],
                                           sc["unit_id"], modality, len(modality), p)
        assert status == 0
        assert np.array_equal(got, want), (U, seed, trial, p)
        assert np.array_equal(mask, wmask), (U, seed, trial, p)
        assert int(kept[0]) == wkept


def test_plan_long_spans():
    """Spans longer than one census step (1,024 slots), with sinks ending on, before and after
    step boundaries and text ranks carried across steps."""
    rng = np.random.default_rng(14)
    units = [sg.grammar_unit(2304, 25, 600), sg.MixedUnit(tuple([1] * 255 + [2] * 2 + [1] * 300)),
             sg.grammar_unit(640, 25, 0), sg.MixedUnit(tuple([3] * 700 + [4] + [3] * 90)),
             sg.grammar_unit(1, 1, 1), (1, 513)]
    lay = sg.build_layout(units, [])
    uid = lay.unit_id.astype(np.int64)
    U = lay.n_units
    length = np.bincount(uid, minlength=U)
    first = np.array([np.nonzero(uid == u)[0][0] for u in range(U)])
    sc = dict(len=length, first=first, last=first + length - 1, flags=np.zeros(U, np.int64))
    for sv, sa, tb in ((255, 1, 650), (256, 2, 0), (257, 0, 10 ** 6), (1, 0, 255), (0, 0, 256),
                       (1021, 3, 1023), (1022, 1, 1025), (1023, 0, 700), (2047, 2, 1500)):
        low = int(rng.integers(0, 2000))
        p = dict(high=low, low=low, recent=0, sv=sv, sa=sa, tb=tb)
        want, wmask, wkept = oracle_plan(sc, lay.modality, p)
        got, mask, kept, status = gpu_plan(length, first, sc["last"], sc["flags"], uid,
                                           lay.modality, lay.n_slots, p)
        assert status == 0 and np.array_equal(got, want) and np.array_equal(mask, wmask)
        assert int(kept[0]) == wkept


def test_plan_several_segments():
    rng = np.random.default_rng(11)
    scs, mods, uids = [], [], []
    n_slots = None
    for _ in range(3):
        while True:
            sc, m = random_layout(rng, 300, hole_p=0.0)
            if n_slots is None or len(m) <= n_slots:
                break
        n_slots = n_slots or len(m) + 50
        scs.append(sc)
        mods.append(np.concatenate([m, np.full(n_slots - len(m), VIDEO)]))
        uids.append(np.concatenate([sc["unit_id"], np.full(n_slots - len(m), -1)]))
    p = dict(high=500, low=400, recent=200, sv=6, sa=3, tb=40)
    cat = lambda key: np.concatenate([s[key] for s in scs])  # noqa: E731
    got, mask, kept, status = gpu_plan(cat("len"), cat("first"), cat("last"), cat("flags"),
                                       np.concatenate(uids), np.concatenate(mods), n_slots, p,
                                       n_seg=3)
    assert status == 0
    for i, sc in enumerate(scs):
        want, wmask, wkept = oracle_plan(sc, mods[i], p)
        assert np.array_equal(got[i * 300:(i + 1) * 300], want)
        assert np.array_equal(mask[i * n_slots:(i + 1) * n_slots], wmask)
        assert int(kept[i]) == wkept


def test_plan_tag_errors():
    rng = np.random.default_rng(12)
    sc, modality = random_layout(rng, 20, hole_p=0.0)
    p = dict(high=0, low=0, recent=10, sv=2, sa=2, tb=5)
    live = np.nonzero(sc["len"] > 0)[0]
    args = lambda d, m: (d["len"], d["first"], d["last"], d["flags"], d["unit_id"], m,  # noqa
                         len(m), p)
    bad = {k: v.copy() for k, v in sc.items()}
    bad["first"][live[3]], bad["first"][live[4]] = sc["first"][live[4]], sc["first"][live[3]]
    bad["last"][live[3]], bad["last"][live[4]] = sc["last"][live[4]], sc["last"][live[3]]
    got, mask, kept, status = gpu_plan(*args(bad, modality))
    assert status == -17 and np.all(got == 0) and np.all(mask == 0) and int(kept[0]) == 0
    bad = {k: v.copy() for k, v in sc.items()}
    bad["last"][live[2]] += 1                            # run longer than its token count
    assert gpu_plan(*args(bad, modality))[3] == -17
    bad = {k: v.copy() for k, v in sc.items()}
    bad["len"][live[-1]] += 10 ** 6                      # unit reaching past the pool
    bad["last"][live[-1]] += 10 ** 6
    assert gpu_plan(*args(bad, modality))[3] == -17
    m2 = modality.copy()
    m2[sc["first"][live[5]] + sc["len"][live[5]] - 1] = 9   # tag out of range inside a unit
    got, mask, kept, status = gpu_plan(*args(sc, m2))
    assert status == -17 and np.all(mask == 0)
    m3 = modality.copy()
    m3[sc["first"][live[5]]] = 4                         # a marker is a valid tag
    assert gpu_plan(*args(sc, m3))[3] == 0


SPAN_PARAMS = {
    "tiny_1p6k_f32": dict(high=600, low=512, sv=8, sa=4, tb=16),
    "single_layer_8k": dict(high=4096, low=4096, sv=64, sa=8, tb=64),
    "history_80k": dict(high=16384, low=16384, sv=256, sa=16, tb=1024),
    "hires_32k_36layer": dict(high=8192, low=6000, sv=256, sa=8, tb=32),
}


def run_span_step(cfg, lay, segs, p, cap_dst=None, rope=None):
    st = make_step(cfg, lay, n_seg=len(segs), cap_dst=cap_dst)
    g = gpu_inputs(lay, segs)
    st.score(g["k_hist"], g["unit_id"], g["modality"])
    st.plan_spans(g["unit_id"], g["modality"], p["low"], p["high"], cfg.recent, p["sv"], p["sa"],
                  p["tb"])
    st.compact_spans(g["k_hist"], g["v_hist"], g["unit_id"], g["modality"], g["pos"],
                     g["k_chunk"], g["v_chunk"], g["chunk_modality"], g["chunk_unit"], rope=rope)
    torch.cuda.synchronize()
    assert int(host(st.d_status)[0]) == 0
    return st


def check_compaction(cfg, lay, seg, st, si, cp, rope_o=None):
    """Every compaction output of segment si against the oracle's result cp."""
    U = st.n_units
    n = cp["n_ctx"]
    assert int(host(st.n_ctx)[si]) == n and int(host(st.n_pages)[si]) == cp["n_pages"]
    cap = st.cap_dst
    tags = slice(si * cap, (si + 1) * cap)
    uid = host(st.unit_id_dst)[tags]
    assert np.array_equal(uid[:n], cp["unit_id"]) and np.all(uid[n:] == -1)
    assert np.array_equal(host(st.modality_dst)[tags][:n], cp["modality"])
    assert np.all(host(st.modality_dst)[tags][n:] == 0)
    assert np.array_equal(host(st.pos_dst)[tags][:n], cp["pos"])
    assert np.all(host(st.pos_dst)[tags][n:] == -1)
    assert np.array_equal(host(st.src_of_dst)[tags][:n], cp["src_of_dst"])
    assert np.all(host(st.src_of_dst)[tags][n:] == -1)
    assert np.array_equal(host(st.unit_remap)[si * U:(si + 1) * U], cp["unit_remap"])
    assert np.array_equal(storage_np(st.v_dst[si])[:n], cp["v"])
    kd = storage_np(st.k_dst[si])[:n]
    if rope_o is None:
        assert np.array_equal(kd, cp["k"])
    else:
        R = rope_o["dims"]
        assert np.array_equal(kd[..., R:], cp["k"][..., R:])
        got = oracle.to_f64(kd, cfg.dtype)[..., :R]
        w = cp["k_f64"][..., :R]
        src = oracle.to_f64(cp["k"], cfg.dtype)
        bound = 0.5 * ulp(w, cfg.dtype) + 2.0 ** -21 * pair_norm(src, R, rope_o["style"])[..., :R]
        assert np.all(np.abs(got - w) <= bound)


def check_span_segment(cfg, lay, seg, st, si, p, rope=None):
    U = lay.n_units
    sl = slice(si * U, (si + 1) * U)
    k = storage_np(seg.k_hist)
    sc = oracle.score_units(k, cfg.dtype, lay.unit_id, lay.modality, cfg.weights, U)
    want, wmask, wkept = oracle_plan(sc, np.asarray(lay.modality), dict(p, recent=cfg.recent))
    assert np.array_equal(host(st.keep_len)[sl], want)
    assert np.array_equal(host(st.keep_slot)[si * lay.n_slots:(si + 1) * lay.n_slots], wmask)
    assert int(host(st.kept_tokens)[si]) == wkept
    rope_o = None
    if rope is not None:
        rope_o = dict(base=rope[0], dims=rope[1], style=("half", "interleaved")[rope[2]],
                      dtype=cfg.dtype)
    cp = oracle.compact_kv(k, storage_np(seg.v_hist), lay.unit_id, lay.modality, lay.pos, None, U,
                           storage_np(seg.k_chunk), storage_np(seg.v_chunk), lay.chunk_modality,
                           lay.chunk_unit, st.cap_dst, st.page_size, rope=rope_o, keep_slot=wmask)
    check_compaction(cfg, lay, seg, st, si, cp, rope_o)
    return cp, want


@pytest.mark.parametrize("cfg_name", ["tiny_1p6k_f32", "single_layer_8k", "history_80k"])
@pytest.mark.parametrize("grammar", [False, True])
def test_span_step_parity(cfg_name, grammar):
    """The workloads as separate units per modality, and grouped into grammar units (each
    second one unit with markers, its frame, its audio and its text)."""
    cfg = sg.CONFIG_BY_NAME[cfg_name]
    stream = sg.make_stream(cfg, grammar=grammar)
    lay, seg = stream.layout, stream.segment(0)
    p = SPAN_PARAMS[cfg_name]
    cap = lay.n_slots + lay.chunk_len if grammar else None
    st = run_span_step(cfg, lay, [seg], p, cap_dst=cap)
    _, kl = check_span_segment(cfg, lay, seg, st, 0, p)
    length = np.bincount(np.asarray(lay.unit_id)[np.asarray(lay.unit_id) >= 0],
                         minlength=lay.n_units)
    assert np.any((kl > 0) & (kl < length)), "the plan must shorten some units"


def test_span_step_three_layers():
    cfg = sg.CONFIG_BY_NAME["hires_32k_36layer"]
    stream = sg.make_stream(cfg, grammar=True)
    lay = stream.layout
    segs = [stream.segment(i) for i in (0, 17, 35)]
    p = SPAN_PARAMS[cfg.name]
    st = run_span_step(cfg, lay, segs, p, cap_dst=lay.n_slots + lay.chunk_len)
    for i, seg in enumerate(segs):
        check_span_segment(cfg, lay, seg, st, i, p)


@pytest.mark.parametrize("cfg_name,rope", [("single_layer_8k", (1.0e6, 128, 0)),
                                           ("tiny_1p6k_f32", (10000.0, 32, 1))])
def test_span_step_with_rope(cfg_name, rope):
    cfg = sg.CONFIG_BY_NAME[cfg_name]
    stream = sg.make_stream(cfg, grammar=True)
    lay, seg = stream.layout, stream.segment(0)
    p = SPAN_PARAMS[cfg_name]
    st = run_span_step(cfg, lay, [seg], p, rope=rope, cap_dst=lay.n_slots + lay.chunk_len)
    check_span_segment(cfg, lay, seg, st, 0, p, rope=rope)


@pytest.mark.parametrize("n_units_extra,shift", [(0, 0), (600, 0), (0, 5)])
def test_compaction_of_arbitrary_masks(n_units_extra, shift):
    """Any per-slot mask (bytes of empty slots set too, values other than 1) against the oracle;
    with 600 extra slotless unit ids the compaction plans through the workspace; the mask may
    start at an odd address."""
    cfg = sg.CONFIG_BY_NAME["single_layer_8k"]
    stream = sg.make_stream(cfg, grammar=True)
    lay, seg = stream.layout, stream.segment(0)
    rng = np.random.default_rng(13)
    U = lay.n_units + n_units_extra
    mask = (rng.random(lay.n_slots) < 0.4).astype(np.uint8) * rng.integers(1, 256, lay.n_slots,
                                                                             dtype=np.uint8)
    uid = np.asarray(lay.unit_id)
    mask[np.isin(uid, rng.choice(lay.n_units, lay.n_units // 3, replace=False))] = 0
    st = make_step(cfg, lay, cap_dst=lay.n_slots + lay.chunk_len, n_units=U)
    g = gpu_inputs(lay, [seg])
    st.score(g["k_hist"], g["unit_id"], g["modality"])
    raw = torch.zeros(len(mask) + 32, dtype=torch.uint8, device="cuda")
    mask_d = raw[shift:shift + len(mask)]
    mask_d.copy_(dev(mask))
    st.compact_spans(g["k_hist"], g["v_hist"], g["unit_id"], g["modality"], g["pos"],
                     g["k_chunk"], g["v_chunk"], g["chunk_modality"], g["chunk_unit"],
                     keep_slot=mask_d)
    torch.cuda.synchronize()
    assert int(host(st.d_status)[0]) == 0
    cp = oracle.compact_kv(storage_np(seg.k_hist), storage_np(seg.v_hist), lay.unit_id,
                           lay.modality, lay.pos, None, U, storage_np(seg.k_chunk),
                           storage_np(seg.v_chunk), lay.chunk_modality, lay.chunk_unit,
                           st.cap_dst, st.page_size, keep_slot=mask)
    check_compaction(cfg, lay, seg, st, 0, cp)


def test_mask_compaction_capacity_error():
    """Kept slots plus the chunk over the destination: E_CAPACITY, no row written, every tag
    row empty."""
    cfg = sg.CONFIG_BY_NAME["single_layer_8k"]
    stream = sg.make_stream(cfg, grammar=True)
    lay, seg = stream.layout, stream.segment(0)
    st = make_step(cfg, lay, cap_dst=1000)
    g = gpu_inputs(lay, [seg])
    st.score(g["k_hist"], g["unit_id"], g["modality"])
    st.k_dst.fill_(3.0)
    st.compact_spans(g["k_hist"], g["v_hist"], g["unit_id"], g["modality"], g["pos"],
                     g["k_chunk"], g["v_chunk"], g["chunk_modality"], g["chunk_unit"],
                     keep_slot=dev(np.ones(lay.n_slots, np.uint8)))
    torch.cuda.synchronize()
    assert int(host(st.d_status)[0]) == -5 and int(host(st.n_ctx)[0]) == 0
    assert np.all(host(st.unit_id_dst) == -1) and np.all(host(st.src_of_dst) == -1)
    assert torch.all(st.k_dst == 3.0)


def test_whole_units_match_the_keep_flag_compaction():
    """A mask of every slot of the selected units gives the whole-unit compaction bit for bit."""
    cfg = sg.CONFIG_BY_NAME["single_layer_8k"]
    stream = sg.make_stream(cfg)
    lay, seg = stream.layout, stream.segment(0)
    st = make_step(cfg, lay)
    g = gpu_inputs(lay, [seg])
    st.score(g["k_hist"], g["unit_id"], g["modality"])
    st.select()
    st.compact(g["k_hist"], g["v_hist"], g["unit_id"], g["modality"], g["pos"], g["k_chunk"],
               g["v_chunk"], g["chunk_modality"], g["chunk_unit"])
    torch.cuda.synchronize()
    ref = {k: getattr(st, k).clone() for k in ("k_dst", "v_dst", "unit_id_dst", "pos_dst",
                                               "src_of_dst", "unit_remap", "n_ctx")}
    uid = g["unit_id"].long()
    mask = ((uid >= 0) & (st.keep.long()[uid.clamp(min=0)] != 0)).to(torch.uint8)
    st.compact_spans(g["k_hist"], g["v_hist"], g["unit_id"], g["modality"], g["pos"],
                     g["k_chunk"], g["v_chunk"], g["chunk_modality"], g["chunk_unit"],
                     keep_slot=mask.contiguous())
    torch.cuda.synchronize()
    for k, v in ref.items():
        assert torch.equal(getattr(st, k), v), k


@pytest.mark.parametrize("shift", [1, 7, 15])
def test_byte_arrays_at_unaligned_addresses(shift):
    """The tag and mask bytes are walked in 16-byte aligned blocks of absolute addresses: the
    plan and the mask compaction give the same result for arrays starting at odd addresses."""
    from paper_2609_34653_amd import omnitide as ot
    rng = np.random.default_rng(40 + shift)
    sc, modality = random_layout(rng, 300, hole_p=0.3)
    n = len(modality)
    p = dict(high=600, low=500, recent=150, sv=5, sa=2, tb=30)
    want, wmask, wkept = oracle_plan(sc, modality, p)
    raw = torch.zeros(n + 64, dtype=torch.uint8, device="cuda")
    mod_odd = raw[shift:shift + n]
    mod_odd.copy_(dev(np.asarray(modality, np.uint8)))
    assert mod_odd.data_ptr() % 16 == shift % 16
    U = len(sc["len"])
    kl = torch.full((U,), -7, dtype=torch.int32, device="cuda")
    ks_raw = torch.full((n + 64,), 7, dtype=torch.uint8, device="cuda")
    ks = ks_raw[shift:shift + n]
    kt = torch.zeros(1, dtype=torch.int32, device="cuda")
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = torch.zeros(ot.omnitide_plan_spans_workspace_bytes(1, n, U), dtype=torch.uint8,
                     device="cuda")
    ot.omnitide_plan_spans(i32(sc["len"]), i32(sc["first"]), i32(sc["last"]), i32(sc["flags"]),
                           i32(sc["unit_id"]), mod_odd, 1, n, U, p["low"], p["high"],
                           p["recent"], p["sv"], p["sa"], p["tb"], kl, ks, kt, ws, st)
    torch.cuda.synchronize()
    assert int(host(st)[0]) == 0
    assert np.array_equal(host(kl), want) and np.array_equal(host(ks), wmask)
    assert int(host(kt)[0]) == wkept
