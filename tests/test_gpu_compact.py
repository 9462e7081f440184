"""HIP compaction (omnitide_compact_kv) vs the oracle, bit for bit, called directly through the C
ABI on layouts built here: every row size the copy kernel specialises (1, 2, 4 and 8 vectors
per thread, a partial row), bf16 and float32, two segments, more than 512 units (the separate
plan kernel, also feeding the rotary copy), and a random keep set with holes between the units.
K/V rows of the destination must equal the oracle's bytes (rotated keys: the rotary bar), and
every tag row (the tail included) its value.
"""
import numpy as np
import pytest
import torch

import oracle
from tests._util import storage_np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_34653_amd import omnitide
    omnitide.lib()
    yield


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def random_layout(rng, n_slots, n_units):
    """Units as contiguous runs in unit order, about 15% of the runs holes; dense positions."""
    uid = np.full(n_slots, -1, np.int32)
    bounds = np.sort(rng.choice(np.arange(1, n_slots), n_units, replace=False))
    for u in range(n_units):
        a = bounds[u - 1] if u else 0
        if rng.random() < 0.85:
            uid[a:bounds[u]] = u
    unit_mod = rng.integers(1, 4, n_units)
    mod = np.where(uid >= 0, unit_mod[np.maximum(uid, 0)], 0).astype(np.uint8)
    pos = np.full(n_slots, -1, np.int32)
    live = uid >= 0
    pos[live] = np.arange(int(live.sum()))
    return uid, mod, pos


def pool(rng, shape, dtype):
    t = torch.from_numpy(rng.standard_normal(shape).astype(np.float32))
    return t.to(torch.bfloat16) if dtype == "bf16" else t


@pytest.mark.parametrize("n_seg,n_slots,H,d,dtype,n_units,L,page", [
    (1, 3000, 3, 64, "f32", 40, 33, 64),      # 768-byte rows: a partial vector per thread
    (2, 2500, 16, 128, "bf16", 50, 70, 128),  # 4 KB rows: two vectors per thread, two segments
    (1, 2000, 16, 128, "f32", 30, 17, 32),    # 8 KB rows: four
    (1, 1200, 32, 128, "f32", 25, 9, 256),    # 16 KB rows: eight
    (1, 6000, 8, 128, "bf16", 600, 100, 64),  # 600 units: the plan kernel, then the copy
])
def test_compact_kv_bit_exact(n_seg, n_slots, H, d, dtype, n_units, L, page):
    run_and_check(n_seg, n_slots, H, d, dtype, n_units, L, page)


@pytest.mark.parametrize("n_seg,n_slots,H,d,dtype,n_units,L,page,rope", [
    (1, 6000, 8, 128, "bf16", 600, 100, 64, (1.0e6, 128, 0)),    # plan kernel, split halves
    (2, 3000, 4, 64, "f32", 700, 40, 32, (10000.0, 48, 1)),     # float32, interleaved, R < d
])
def test_compact_kv_rope_plan_kernel(n_seg, n_slots, H, d, dtype, n_units, L, page, rope):
    """Rotary compaction with more than 512 units (the separate plan kernel feeds the rotary
    copy): tags, V rows, chunk rows, unshifted rows and dimensions past the rotary width
    bit-exact; rotated elements at the rotary parity bar."""
    run_and_check(n_seg, n_slots, H, d, dtype, n_units, L, page, rope)


def run_and_check(n_seg, n_slots, H, d, dtype, n_units, L, page, rope=None):
    from paper_2609_34653_amd import omnitide as ot
    rng = np.random.default_rng(n_slots + n_units + H)
    lays = [random_layout(rng, n_slots, n_units) for _ in range(n_seg)]
    keeps = [(rng.random(n_units) < 0.6).astype(np.uint8) for _ in range(n_seg)]
    k_src = torch.stack([pool(rng, (n_slots, H, d), dtype) for _ in range(n_seg)])
    v_src = torch.stack([pool(rng, (n_slots, H, d), dtype) for _ in range(n_seg)])
    k_chunk = torch.stack([pool(rng, (L, H, d), dtype) for _ in range(n_seg)])
    v_chunk = torch.stack([pool(rng, (L, H, d), dtype) for _ in range(n_seg)])
    chunk_mod = rng.integers(1, 4, L).astype(np.uint8)
    chunk_unit = (np.arange(L) * min(3, L) // L).astype(np.int32)   # units 0.. in order
    # score-side inputs of the call, from the tags (plain host arithmetic)
    unit_len = np.zeros((n_seg, n_units), np.int32)
    unit_first = np.full((n_seg, n_units), n_slots, np.int32)
    for s, (uid, _, _) in enumerate(lays):
        live = np.nonzero(uid >= 0)[0]
        unit_len[s] = np.bincount(uid[live], minlength=n_units)
        for u in np.unique(uid[live])[::-1]:
            unit_first[s, u] = live[uid[live] == u][0]
    kept = [int(unit_len[s][keeps[s] != 0].sum()) for s in range(n_seg)]
    cap = max(kept) + L + 37
    dt = k_src.dtype
    k_dst = torch.full((n_seg, cap, H, d), float("nan"), dtype=dt, device="cuda")
    v_dst = torch.full_like(k_dst, float("nan"))
    i32 = dict(dtype=torch.int32, device="cuda")
    uid_dst = torch.full((n_seg * cap,), 77, **i32)
    mod_dst = torch.full((n_seg * cap,), 9, dtype=torch.uint8, device="cuda")
    pos_dst = torch.full((n_seg * cap,), 77, **i32)
    src_dst = torch.full((n_seg * cap,), 77, **i32)
    remap = torch.full((n_seg * n_units,), 77, **i32)
    n_ctx = torch.full((n_seg,), 77, **i32)
    n_pages = torch.full((n_seg,), 77, **i32)
    ws = torch.full((max(1, ot.omnitide_compact_workspace_bytes(n_seg, n_units, cap)),), 0xFF,
                    dtype=torch.uint8, device="cuda")
    st = torch.zeros(1, **i32)
    args = (k_src.cuda(), v_src.cuda(), page, dev(np.concatenate([x[0] for x in lays])),
            dev(np.concatenate([x[1] for x in lays])), dev(np.concatenate([x[2] for x in lays])),
            dev(np.concatenate(keeps)), dev(unit_len.ravel()), dev(unit_first.ravel()), n_units,
            k_chunk.cuda(), v_chunk.cuda(), dev(chunk_mod), dev(chunk_unit), k_dst, v_dst,
            uid_dst, mod_dst, pos_dst, src_dst, remap, n_ctx, n_pages, ws)
    if rope is None:
        ot.omnitide_compact_kv(*args, st)
    else:
        ot.omnitide_compact_kv_rope(*args, rope[0], rope[1], rope[2], d_status=st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    kd, vd = storage_np(k_dst), storage_np(v_dst)
    tags = {nm: t.cpu().numpy().reshape(n_seg, -1)
            for nm, t in (("unit_id", uid_dst), ("modality", mod_dst), ("pos", pos_dst),
                          ("src_of_dst", src_dst), ("unit_remap", remap))}
    for s in range(n_seg):
        uid, mod, pos = lays[s]
        style = None if rope is None else ("half", "interleaved")[rope[2]]
        cp = oracle.compact_kv(storage_np(k_src[s]), storage_np(v_src[s]), uid, mod, pos,
                               keeps[s], n_units, storage_np(k_chunk[s]), storage_np(v_chunk[s]),
                               chunk_mod, chunk_unit, cap, page,
                               rope=None if rope is None else
                               dict(base=rope[0], dims=rope[1], style=style, dtype=dtype))
        n = cp["n_ctx"]
        assert n == kept[s] + L
        assert int(n_ctx[s]) == n and int(n_pages[s]) == cp["n_pages"]
        assert np.array_equal(vd[s][:n], cp["v"])
        if rope is None:
            assert np.array_equal(kd[s][:n], cp["k"])
        else:
            check_rotated(kd[s][:n], cp, pos, dtype, rope[1], style)
        for nm in ("unit_id", "modality", "pos", "src_of_dst"):
            assert np.array_equal(tags[nm][s][:n].astype(np.int64), cp[nm].astype(np.int64)), nm
        assert np.all(tags["unit_id"][s][n:] == -1) and np.all(tags["modality"][s][n:] == 0)
        assert np.all(tags["pos"][s][n:] == -1) and np.all(tags["src_of_dst"][s][n:] == -1)
        assert np.array_equal(tags["unit_remap"][s].astype(np.int64), cp["unit_remap"])


def check_rotated(got_bits, cp, pos_src, dtype, rot_dims, style):
    """Rotary compaction bar (as in test_gpu_rope): rows whose position does not change and
    dimensions past the rotary width bit-exact; rotated elements within half an ulp of the exact
    rotation plus 2^-21 of their pair's length."""
    from tests.test_gpu_rope import pair_norm, ulp
    n = got_bits.shape[0]
    shift = np.zeros(n, np.int64)
    kept = cp["kept"]
    shift[:kept] = cp["pos"][:kept] - np.asarray(pos_src)[cp["src_of_dst"][:kept]]
    assert np.any(shift != 0), "the layout must move some rows"
    same = shift == 0
    assert np.array_equal(got_bits[same], cp["k"][same])
    assert np.array_equal(got_bits[..., rot_dims:], cp["k"][..., rot_dims:])
    got = oracle.to_f64(got_bits, dtype)[~same][..., :rot_dims]
    want = cp["k_f64"][~same][..., :rot_dims]
    src = oracle.to_f64(cp["k"], dtype)[~same]
    bound = 0.5 * ulp(want, dtype) + 2.0 ** -21 * pair_norm(src, rot_dims, style)[..., :rot_dims]
    assert np.all(np.abs(got - want) <= bound)
