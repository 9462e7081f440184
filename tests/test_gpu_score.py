"""HIP unit scoring (omnitide_score_units) vs the oracle, bit for bit, called directly through the
C ABI: every row width the kernel specialises (16-byte vectors per lane 1, 2, 4, 8 and 16,
full and partial), bf16 and float32 pools, two segments, units as runs with holes and units
scattered over the pool, special key values (NaN, infinities, subnormals, zeros, values past
the clamp), and both load-batch depths (small grids, and grids of at least 4,096 waves).
"""
import numpy as np
import pytest
import torch

import oracle
import streamgen as sg
from tests._util import storage_np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_34653_amd import omnitide
    omnitide.lib()
    yield


def random_tags(rng, n_slots, n_units, scattered):
    """Unit ids and modalities: contiguous runs with holes, or ids scattered over the slots."""
    if scattered:
        uid = rng.integers(-1, n_units, n_slots)
    else:
        uid = np.full(n_slots, -1)
        bounds = np.sort(rng.choice(np.arange(1, n_slots), n_units, replace=False))
        for u in range(n_units):
            a = bounds[u - 1] if u else 0
            b = bounds[u]
            if rng.random() < 0.85:
                uid[a:b] = u
    unit_mod = rng.integers(0, 4, n_units)
    mod = np.where(uid >= 0, unit_mod[np.maximum(uid, 0)], rng.integers(0, 4, n_slots))
    return uid.astype(np.int32), mod.astype(np.uint8)


def random_keys(rng, shape, dtype):
    x = rng.standard_normal(shape) * rng.choice([0.01, 1.0, 40.0], shape, p=[0.2, 0.7, 0.1])
    special = rng.random(shape) < 0.01
    x = np.where(special, rng.choice([np.nan, np.inf, -np.inf, 0.0, 1e-40, 1e30], shape), x)
    t = torch.from_numpy(np.ascontiguousarray(x, np.float32))
    return t.to(torch.bfloat16) if dtype == "bf16" else t


@pytest.mark.parametrize("n_seg,n_slots,H,d,dtype,n_units,scattered", [
    (1, 3000, 3, 64, "f32", 40, False),     # 48 vectors per row: one per lane, partial
    (2, 2000, 5, 128, "bf16", 25, False),   # 80 vectors: two per lane, partial
    (1, 1500, 8, 128, "f32", 60, False),    # 256 vectors: four per lane
    (1, 1000, 16, 128, "bf16", 30, True),   # 256 vectors, units scattered over the pool
    (1, 900, 32, 128, "bf16", 20, False),   # 512 vectors: eight per lane
    (1, 700, 12, 128, "f32", 9, False),     # 384 vectors: eight per lane, partial
    (1, 600, 32, 128, "f32", 12, True),     # 1,024 vectors: sixteen per lane
    # grids of at least 4,096 waves take the one-row batches (the 80K and 36-layer workloads)
    (4, 16384, 3, 64, "f32", 200, False),   # 48 vectors per row, partial, shallow batches
    (2, 32768, 8, 128, "f32", 300, True),   # 256 vectors: four per lane, shallow batches
])
def test_score_units_bit_exact(n_seg, n_slots, H, d, dtype, n_units, scattered):
    from paper_2609_34653_amd import omnitide as ot
    rng = np.random.default_rng(n_slots + H + d)
    k = torch.stack([random_keys(rng, (n_slots, H, d), dtype) for _ in range(n_seg)])
    tags = [random_tags(rng, n_slots, n_units, scattered) for _ in range(n_seg)]
    uid = np.stack([t[0] for t in tags])
    mod = np.stack([t[1] for t in tags])
    nu = n_seg * n_units
    out = dict(wsum=torch.full((nu,), -7, dtype=torch.int64, device="cuda"),
               len=torch.full((nu,), -7, dtype=torch.int32, device="cuda"),
               first=torch.full((nu,), -7, dtype=torch.int32, device="cuda"),
               last=torch.full((nu,), -7, dtype=torch.int32, device="cuda"),
               flags=torch.full((nu,), -7, dtype=torch.int32, device="cuda"))
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    ot.omnitide_score_units(k.cuda(), torch.from_numpy(uid).cuda(), torch.from_numpy(mod).cuda(),
                            sg.DEFAULT_WEIGHTS, n_units, out["wsum"], out["len"], out["first"],
                            out["last"], out["flags"], st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    got = {key: t.cpu().numpy().reshape(n_seg, n_units) for key, t in out.items()}
    for s in range(n_seg):
        want = oracle.score_units(storage_np(k[s]), dtype, uid[s], mod[s], sg.DEFAULT_WEIGHTS,
                                  n_units)
        for key in ("wsum", "len", "first", "last", "flags"):
            assert np.array_equal(got[key][s].astype(np.int64), want[key]), (s, key)
