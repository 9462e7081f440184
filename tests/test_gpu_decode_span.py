"""HIP decode attention over a pool with holes (native and ordered-suffix layouts) vs the float64
oracle's span attention with the decode tokens as queries, through the C ABI.

Bar: max |err| <= 2e-5 and mean |err| <= 2e-6 over every output element, as for the decode over
the compacted pool (probabilities enter the products with about 16 significant bits).
"""
import numpy as np
import pytest
import torch

import oracle
from tests._util import storage_np
from tests.test_gpu_native import native_80k, random_span_pool
from tests.test_gpu_parity import dev, host

pytestmark = pytest.mark.gpu

MAX_ABS, MEAN_ABS = 2e-5, 2e-6


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_34653_amd import omnitide
    omnitide.lib()
    yield


def bf16(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(torch.bfloat16)


def run_decode_span(q, k, v, key_pos, span, q_pos0, scale, skip=True, expect_status=0):
    """q [n_seg, n_q, Hq, d], k/v [n_seg, cap, Hkv, d] (CPU bf16); key_pos [n_seg, cap].
    skip: True (tile skipping), False (the full span) or "pos" (position order)."""
    from paper_2609_34653_amd import omnitide as ot
    n_seg, nq, Hq, d = q.shape
    cap, Hkv = k.shape[1], k.shape[2]
    nb = ot.omnitide_decode_span_workspace_bytes(n_seg, cap, nq, Hq, Hkv, d)
    ws = torch.full((nb // 4 + 1,), float("nan"), device="cuda").view(torch.uint8)[:nb]
    out = torch.full((n_seg, nq, Hq, d), float("nan"), device="cuda")
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    ot.omnitide_decode_span_attn(q.cuda().contiguous(), k.cuda().contiguous(),
                                 v.cuda().contiguous(),
                                 dev(np.asarray(key_pos, np.int32).reshape(-1)),
                                 dev(np.asarray(span, np.int32)),
                                 dev(np.asarray(q_pos0, np.int32)), scale, out, ws, st,
                                 skip_empty_tiles=skip is True, position_order=skip == "pos")
    torch.cuda.synchronize()
    assert int(host(st)[0]) == expect_status
    return host(out)


def check(out, q, k, v, key_pos, span, q_pos0, scale):
    f = lambda t: oracle.to_f64(storage_np(t), "bf16")  # noqa: E731
    occ = np.nonzero(np.asarray(key_pos)[:span] >= 0)[0]      # only entries can be visible
    ref = oracle.span_attention(f(q), f(k[occ]), f(v[occ]), np.asarray(key_pos)[occ], len(occ),
                                q_pos0, scale)
    err = np.abs(out.astype(np.float64) - ref)
    assert np.isfinite(out).all()
    assert err.max() <= MAX_ABS, err.max()
    assert err.mean() <= MEAN_ABS, err.mean()


@pytest.mark.parametrize("cap,nq,Hq,Hkv,d,fill,seed,skip", [
    (700, 1, 32, 8, 128, 0.5, 0, True),       # ragged span, GQA 4
    (700, 1, 32, 8, 128, 0.5, 0, False),      # the same, every tile of the span read
    (3000, 2, 16, 4, 128, 0.3, 1, True),      # two tokens, 8 query vectors per KV head
    (5000, 1, 8, 1, 64, 0.1, 2, True),        # sparse, many empty tiles, d = 64
    (5000, 1, 8, 1, 64, 0.1, 2, False),
    (1500, 4, 8, 4, 128, 0.95, 3, True),      # nearly full, four tokens
    (9000, 1, 4, 4, 64, 0.6, 4, False),       # no grouping
    (700, 1, 32, 8, 128, 0.5, 0, "pos"),      # position order: the same pools
    (3000, 2, 16, 4, 128, 0.3, 1, "pos"),
    (5000, 1, 8, 1, 64, 0.1, 2, "pos"),
    (1500, 4, 8, 4, 128, 0.95, 3, "pos"),
    (9000, 1, 4, 4, 64, 0.6, 4, "pos"),
    (300, 1, 8, 1, 128, 0.02, 11, "pos"),     # a handful of entries (fewer than one block)
])
def test_decode_span_random_pools(cap, nq, Hq, Hkv, d, fill, seed, skip):
    rng = np.random.default_rng(seed)
    k, v, key_pos, span, q_pos0 = random_span_pool(rng, cap, nq, Hkv, d, fill)
    q = bf16(rng.standard_normal((nq, Hq, d)))
    scale = d ** -0.5
    out = run_decode_span(q[None], k[None], v[None], key_pos[None], [span], [q_pos0], scale,
                          skip=skip)
    check(out[0], q, k, v, key_pos, span, q_pos0, scale)


def test_decode_span_several_segments():
    rng = np.random.default_rng(5)
    cap, nq, Hq, Hkv, d = 2600, 1, 32, 8, 128
    pools = [random_span_pool(rng, cap, nq, Hkv, d, f) for f in (0.05, 0.6, 0.97)]
    q = bf16(rng.standard_normal((3, nq, Hq, d)))
    for skip in (True, False, "pos"):
        out = run_decode_span(q, torch.stack([p[0] for p in pools]),
                              torch.stack([p[1] for p in pools]),
                              np.stack([p[2] for p in pools]), [p[3] for p in pools],
                              [p[4] for p in pools], 0.09, skip=skip)
        for i, (k, v, kp, span, qp) in enumerate(pools):
            check(out[i], q[i], k, v, kp, span, qp, 0.09)


def test_decode_span_dense_positions_match_decode():
    """key_pos = slot index and q_pos0 = span - n_q: the decode over the compacted pool."""
    from paper_2609_34653_amd import omnitide as ot
    rng = np.random.default_rng(6)
    cap, nq, Hq, Hkv, d, n = 4000, 2, 8, 2, 128, 3333
    k = bf16(rng.standard_normal((1, cap, Hkv, d)))
    v = bf16(rng.standard_normal((1, cap, Hkv, d)))
    q = bf16(rng.standard_normal((1, nq, Hq, d)))
    kp = np.where(np.arange(cap) < n, np.arange(cap), -1)
    out = run_decode_span(q, k, v, kp[None], [n], [n - nq], 0.09)
    ref = torch.zeros(1, nq, Hq, d, device="cuda")
    nb = ot.omnitide_decode_workspace_bytes(1, cap, nq, Hq, Hkv, d)
    ws = torch.zeros(max(nb, 1), dtype=torch.uint8, device="cuda")
    ot.omnitide_decode_attn(q.cuda(), k.cuda(), v.cuda(), dev(np.array([n], np.int32)), 0.09,
                            ref, ws)
    torch.cuda.synchronize()
    assert np.abs(out - host(ref)).max() <= 2e-6
    check(out[0], q[0], k[0], v[0], kp, n, n - nq, 0.09)


def decode_compacted(q, k, v, key_pos, n, scale):
    """omnitide_decode_attn over the entries of a holey pool moved to slots 0 .. n-1 in position
    order (the same capacity, so the same split count)."""
    from paper_2609_34653_amd import omnitide as ot
    n_seg, cap, Hkv, d = k.shape
    nq, Hq = q.shape[1], q.shape[2]
    kc, vc = torch.zeros_like(k), torch.zeros_like(v)
    for i in range(n_seg):
        slots = np.argsort(np.where(key_pos[i] >= 0, key_pos[i], np.iinfo(np.int64).max),
                           kind="stable")[:n[i]]
        assert np.array_equal(key_pos[i][slots], np.arange(n[i]))
        kc[i, :n[i]] = k[i, torch.from_numpy(slots)]
        vc[i, :n[i]] = v[i, torch.from_numpy(slots)]
    out = torch.zeros(n_seg, nq, Hq, d, device="cuda")
    nb = ot.omnitide_decode_workspace_bytes(n_seg, cap, nq, Hq, Hkv, d)
    ws = torch.zeros(max(nb, 1), dtype=torch.uint8, device="cuda")
    ot.omnitide_decode_attn(q.cuda(), kc.cuda(), vc.cuda(), dev(np.asarray(n, np.int32)), scale,
                            out, ws)
    torch.cuda.synchronize()
    return host(out)


@pytest.mark.parametrize("cap,nq,Hq,Hkv,d,fills,seed", [
    (6000, 1, 32, 8, 128, (0.4,), 12),
    (2500, 2, 8, 2, 64, (0.15, 0.8), 13),     # two segments, two tokens, d = 64
])
def test_decode_position_order_bitwise_equals_compacted(cap, nq, Hq, Hkv, d, fills, seed):
    """Position order reads the same keys in the same blocks as the decode over the compacted
    pool: the outputs agree bit for bit."""
    rng = np.random.default_rng(seed)
    pools = [random_span_pool(rng, cap, nq, Hkv, d, f, nan_holes=False) for f in fills]
    q = bf16(rng.standard_normal((len(fills), nq, Hq, d)))
    k, v = torch.stack([p[0] for p in pools]), torch.stack([p[1] for p in pools])
    kp = np.stack([p[2] for p in pools])
    out = run_decode_span(q, k, v, kp, [p[3] for p in pools], [p[4] for p in pools], 0.08,
                          skip="pos")
    ref = decode_compacted(q, k, v, kp, [p[4] + nq for p in pools], 0.08)
    assert np.array_equal(out, ref)


def test_decode_position_order_errors_reported():
    """Entries that are not the positions 0 .. q_pos0 + n_q - 1 once each: OMNITIDE_E_TAGS."""
    rng = np.random.default_rng(14)
    k, v, kp, span, qp = random_span_pool(rng, 1500, 1, 2, 128, 0.5, nan_holes=False)
    q = bf16(rng.standard_normal((1, 1, 8, 128)))
    hist = np.nonzero((kp >= 0) & (kp < qp))[0]
    run = lambda kp2, qp2=qp, st=-17: run_decode_span(  # noqa: E731
        q, k[None], v[None], kp2[None], [span], [qp2], 0.1, skip="pos", expect_status=st)
    run(kp, st=0)
    dup = kp.copy()
    dup[hist[2]] = kp[hist[9]]
    run(dup)
    gone = kp.copy()
    gone[hist[4]] = -1
    run(gone)
    run(kp, qp2=-1)
    run(kp, qp2=qp + 1)


def test_decode_span_native_80k():
    """The last token of the chunk decodes over the 80K history evicted in place (the chunk in
    a hole, the span past 60K slots), in all three traversals; position order equals the
    decode over the compacted pool bit for bit."""
    cfg, q, k, v, key_pos, span, q_pos0, s0 = native_80k()
    L = q.shape[0]
    qd = q[L - 1:L]
    for skip in (True, False, "pos"):
        out = run_decode_span(qd[None], k[None], v[None], key_pos[None], [span],
                              [q_pos0 + L - 1], cfg.scale, skip=skip)
        check(out[0], qd, k, v, key_pos, span, q_pos0 + L - 1, cfg.scale)
    ref = decode_compacted(qd[None], k[None], v[None], key_pos[None], [q_pos0 + L], cfg.scale)
    assert np.array_equal(out, ref)


def test_decode_span_capacity_error():
    rng = np.random.default_rng(9)
    k, v, kp, span, qp = random_span_pool(rng, 500, 1, 2, 64, 0.5, nan_holes=False)
    q = bf16(rng.standard_normal((1, 1, 4, 64)))
    out = run_decode_span(q, k[None], v[None], kp[None], [501], [qp], 0.1, expect_status=-5)
    assert np.isnan(out).all()                     # the segment's output is not written
