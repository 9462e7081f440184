"""HIP chunk attention (omnitide_chunk_attn) vs the float64 oracle, called directly through the C
ABI on pools built here: ragged tiles and tails, several segments and splits, d = 64 and 128,
grouping 1 to 8, no history, a single query, and scores that keep rising along the keys so that
the softmax reference has to move on later tiles (the kernel's slow path).

Bar: max |err| <= 1e-2 and mean |err| <= 1e-3 of the float64 oracle on the same bf16 inputs.
"""
import numpy as np
import pytest
import torch

import oracle
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


def bf16(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(torch.bfloat16)


def run_attn(q, k, v, n_ctx, scale):
    """q [n_seg, L, Hq, d], k/v [n_seg, cap, Hkv, d] (bf16, host); returns out [n_seg, L, Hq, d]
    float32 and the device status."""
    from paper_2609_34653_amd import omnitide as ot
    n_seg, L, Hq, d = q.shape
    cap, Hkv = k.shape[1], k.shape[2]
    out = torch.full((n_seg, L, Hq, d), float("nan"), device="cuda")
    nb = ot.omnitide_attn_workspace_bytes(n_seg, cap, L, Hq, Hkv, d)
    ws = torch.full((max(nb, 1),), 0xFF, dtype=torch.uint8, device="cuda")   # NaN-filled
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    ot.omnitide_chunk_attn(q.cuda(), k.cuda(), v.cuda(),
                           torch.tensor(n_ctx, dtype=torch.int32, device="cuda"), scale, out, ws,
                           st)
    torch.cuda.synchronize()
    return out.cpu().numpy(), int(st.item())


def check(out, q, k, v, n, scale):
    f = lambda t: oracle.to_f64(storage_np(t), "bf16")  # noqa: E731
    want = oracle.chunk_attention(f(q), f(k)[:n], f(v)[:n], scale)
    err = np.abs(out - want)
    assert np.all(np.isfinite(out))
    assert err.max() <= MAX_ABS and err.mean() <= MEAN_ABS, (err.max(), err.mean())
    return err


@pytest.mark.parametrize("n_ctx,cap,L,Hq,Hkv,d,scale", [
    ([700], 1000, 37, 8, 2, 128, None),            # ragged tiles and row tile, grouping 4
    ([4000, 1300], 4096, 200, 16, 4, 64, None),   # two segments, several splits, d = 64
    ([665], 700, 665, 32, 8, 128, None),          # no history: the chunk attends to itself
    ([2049], 2100, 1, 32, 8, 128, None),          # a single query over a ragged tail
    ([3000], 3100, 64, 8, 8, 128, 0.05),          # no grouping, small scale
    ([5000], 5000, 129, 32, 8, 128, 2.0),         # large scores, n_ctx = cap
])
def test_chunk_attention_parity(n_ctx, cap, L, Hq, Hkv, d, scale):
    rng = np.random.default_rng(sum(n_ctx) + L)
    n_seg = len(n_ctx)
    q = bf16(rng.standard_normal((n_seg, L, Hq, d)))
    k = bf16(rng.standard_normal((n_seg, cap, Hkv, d)))
    v = bf16(rng.standard_normal((n_seg, cap, Hkv, d)))
    scale = d ** -0.5 if scale is None else scale
    out, status = run_attn(q, k, v, n_ctx, scale)
    assert status == 0
    for s, n in enumerate(n_ctx):
        check(out[s], q[s], k[s], v[s], n, scale)


def test_chunk_attention_rising_scores_move_the_reference():
    """Key j is alpha_j * u with alpha_j rising linearly and every query close to u, so each
    64-key tile's scores exceed the previous tiles' by far more than 32 in log2 units: the
    reference taken from the first tile would overflow the tile sums, and the kernel must move
    it again and again.  The result is dominated by the last visible keys."""
    rng = np.random.default_rng(17)
    n, L, Hq, Hkv, d = 1500, 40, 8, 2, 128
    u = rng.standard_normal(d)
    u /= np.linalg.norm(u)
    scale = d ** -0.5
    # scale * alpha * <q, u> * log2(e) grows by ~1 per key: ~64 per tile
    alpha = np.arange(n) / (scale * np.log2(np.e))
    k = alpha[:, None, None] * u[None, None, :] + 0.01 * rng.standard_normal((n, Hkv, d))
    q = u[None, None, :] + 0.01 * rng.standard_normal((L, Hq, d))
    v = rng.standard_normal((n, Hkv, d))
    out, status = run_attn(bf16(q)[None], bf16(k)[None], bf16(v)[None], [n], scale)
    assert status == 0
    check(out[0], bf16(q), bf16(k), bf16(v), n, scale)


def run_attn_dtypes(q, k, v, n_ctx, scale, out_dtype):
    """Like run_attn, with q/k/v of any storage dtype (host tensors) and the output dtype."""
    from paper_2609_34653_amd import omnitide as ot
    n_seg, L, Hq, d = q.shape
    cap, Hkv = k.shape[1], k.shape[2]
    dt = ot.F32 if q.dtype == torch.float32 else ot.BF16
    out = torch.full((n_seg, L, Hq, d), float("nan"), dtype=out_dtype, device="cuda")
    nb = ot.omnitide_attn_workspace_bytes(n_seg, cap, L, Hq, Hkv, d, dtype=dt)
    ws = torch.full((max(nb, 1),), 0xFF, dtype=torch.uint8, device="cuda")
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    ot.omnitide_chunk_attn(q.cuda(), k.cuda(), v.cuda(),
                           torch.tensor(n_ctx, dtype=torch.int32, device="cuda"), scale, out, ws,
                           st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    return out.cpu()


@pytest.mark.parametrize("n_ctx,cap,L,Hq,Hkv,d", [
    ([17048], 17100, 665, 32, 8, 128),        # the 80K-history shape: three splits, combine
    ([700, 300], 800, 37, 8, 2, 64),          # two segments, one split
])
def test_output_and_input_dtypes(n_ctx, cap, L, Hq, Hkv, d):
    """bf16 output: the float32 result rounded to nearest even, bit for bit (single-split and
    combine paths).  float32 inputs: rounded to bf16 inside the library, so the output equals the
    call on bf16 copies rounded the same way (torch's cast), bit for bit."""
    rng = np.random.default_rng(77)
    n_seg = len(n_ctx)
    q32 = torch.from_numpy(rng.standard_normal((n_seg, L, Hq, d)).astype(np.float32))
    k32 = torch.from_numpy(rng.standard_normal((n_seg, cap, Hkv, d)).astype(np.float32))
    v32 = torch.from_numpy(rng.standard_normal((n_seg, cap, Hkv, d)).astype(np.float32))
    q, k, v = (t.to(torch.bfloat16) for t in (q32, k32, v32))
    scale = d ** -0.5
    ref = run_attn_dtypes(q, k, v, n_ctx, scale, torch.float32)
    for i, n in enumerate(n_ctx):
        check(ref[i].numpy(), q[i], k[i], v[i], n, scale)
    ob = run_attn_dtypes(q, k, v, n_ctx, scale, torch.bfloat16)
    assert torch.equal(ob.view(torch.int16), ref.to(torch.bfloat16).view(torch.int16))
    of = run_attn_dtypes(q32, k32, v32, n_ctx, scale, torch.float32)
    assert torch.equal(of, ref)
    ofb = run_attn_dtypes(q32, k32, v32, n_ctx, scale, torch.bfloat16)
    assert torch.equal(ofb.view(torch.int16), ob.view(torch.int16))
