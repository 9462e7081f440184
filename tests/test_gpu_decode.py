"""HIP decode attention vs the float64 oracle (the chunk-attention definition with the last n_q
tokens as queries), through the C ABI.

Bar: max |err| <= 2e-5 and mean |err| <= 2e-6 -- the kernel keeps the probabilities in float
(only bf16 inputs), so the error is float accumulation error, far inside the prefill bar.
"""
import numpy as np
import pytest
import torch

import oracle
from tests._util import storage_np

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


def run_decode(n_ctx, cap, n_q, Hq, Hkv, d, seed=0, scale=None):
    from paper_2609_34653_amd import omnitide as ot
    rng = np.random.default_rng(seed)
    n_seg = len(n_ctx)
    q = bf16(rng.standard_normal((n_seg, n_q, Hq, d)))
    k = bf16(rng.standard_normal((n_seg, cap, Hkv, d)))
    v = bf16(rng.standard_normal((n_seg, cap, Hkv, d)))
    scale = d ** -0.5 if scale is None else scale
    out = torch.full((n_seg, n_q, Hq, d), float("nan"), device="cuda")
    nb = ot.omnitide_decode_workspace_bytes(n_seg, cap, n_q, Hq, Hkv, d)
    ws = torch.zeros(max(nb, 1), dtype=torch.uint8, device="cuda")
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    ot.omnitide_decode_attn(q.cuda(), k.cuda(), v.cuda(),
                            torch.tensor(n_ctx, dtype=torch.int32, device="cuda"), scale, out,
                            ws, st)
    torch.cuda.synchronize()
    return q, k, v, out.cpu().numpy(), int(st.item()), scale


def oracle_decode(q, k, v, n, scale):
    f = lambda t: oracle.to_f64(storage_np(t), "bf16")  # noqa: E731
    return oracle.chunk_attention(f(q), f(k)[:n], f(v)[:n], scale)


@pytest.mark.parametrize("n_ctx,cap,n_q,Hq,Hkv,d", [
    ([1], 64, 1, 32, 8, 128),                 # a single visible key
    ([777], 1000, 1, 32, 8, 128),             # ragged, several splits
    ([5000, 63, 2048], 5000, 2, 16, 8, 128),  # several segments, n_ctx = cap and tiny
    ([3001], 3001, 1, 8, 1, 64),              # 8 query heads on one KV head, d = 64
    ([1500, 1499], 2000, 2, 8, 8, 64),        # no grouping, two tokens
    ([16948], 17049, 1, 32, 8, 128),          # the 80K-history pool after compaction
    ([2500, 700], 2600, 2, 32, 8, 128),       # eight query vectors per KV head, d = 128
    ([129], 129, 4, 8, 4, 64),                # four tokens (causal among them), eight vectors
])
def test_decode_parity(n_ctx, cap, n_q, Hq, Hkv, d):
    q, k, v, out, status, scale = run_decode(n_ctx, cap, n_q, Hq, Hkv, d)
    assert status == 0
    for s, n in enumerate(n_ctx):
        want = oracle_decode(q[s], k[s], v[s], n, scale)
        err = np.abs(out[s] - want)
        assert err.max() <= MAX_ABS and err.mean() <= MEAN_ABS, (s, err.max(), err.mean())


def test_decode_large_scores_stay_finite():
    """Scores far from zero (a large scale) exercise the running maximum."""
    q, k, v, out, status, scale = run_decode([900], 1024, 1, 32, 8, 128, seed=3, scale=2.0)
    assert status == 0 and np.all(np.isfinite(out))
    want = oracle_decode(q[0], k[0], v[0], 900, scale)
    assert np.abs(out[0] - want).max() <= 1e-3


def test_decode_capacity_error_on_device():
    """A segment whose n_ctx exceeds the pool reports OMNITIDE_E_CAPACITY and is not written;
    the other segments are still correct."""
    q, k, v, out, status, scale = run_decode([300, 5000], 1000, 1, 32, 8, 128, seed=5)
    assert status == -5
    assert np.all(np.isnan(out[1]))
    want = oracle_decode(q[0], k[0], v[0], 300, scale)
    assert np.abs(out[0] - want).max() <= MAX_ABS


def test_decode_workspace_reused_across_shapes():
    """One workspace serves calls of different shapes and split counts in a row (each call's
    partials overwrite what the previous one left)."""
    from paper_2609_34653_amd import omnitide as ot
    cases = [([16948], 17049, 1, 32, 8, 128), ([2999], 3000, 1, 32, 8, 128),
             ([5000, 63, 2048], 5000, 2, 16, 8, 128), ([40], 4000, 1, 8, 2, 64),
             ([16948], 17049, 1, 32, 8, 128)]
    need = max(ot.omnitide_decode_workspace_bytes(len(n), c, nq, hq, hkv, d)
               for n, c, nq, hq, hkv, d in cases)
    ws = torch.full((need,), 0xFF, dtype=torch.uint8, device="cuda")   # NaN-filled
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    for i, (n_ctx, cap, n_q, Hq, Hkv, d) in enumerate(cases):
        rng = np.random.default_rng(40 + i)
        n_seg = len(n_ctx)
        q = bf16(rng.standard_normal((n_seg, n_q, Hq, d)))
        k = bf16(rng.standard_normal((n_seg, cap, Hkv, d)))
        v = bf16(rng.standard_normal((n_seg, cap, Hkv, d)))
        out = torch.full((n_seg, n_q, Hq, d), float("nan"), device="cuda")
        ot.omnitide_decode_attn(q.cuda(), k.cuda(), v.cuda(),
                                torch.tensor(n_ctx, dtype=torch.int32, device="cuda"),
                                d ** -0.5, out, ws, st)
        torch.cuda.synchronize()
        assert int(st.item()) == 0
        got = out.cpu().numpy()
        for s, n in enumerate(n_ctx):
            err = np.abs(got[s] - oracle_decode(q[s], k[s], v[s], n, d ** -0.5))
            assert err.max() <= MAX_ABS and err.mean() <= MEAN_ABS, (i, s, err.max())
