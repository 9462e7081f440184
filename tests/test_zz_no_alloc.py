"""The allocation-free chunk attention (split-KV partials in the library's fixed scratch)
against the workspace entry point, through the C ABI: bitwise equal outputs on calls in a row,
each smaller than the one before, and a final call that needs no scratch at all."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_34653_amd import omnitide
    omnitide.lib()
    yield


def inputs(seed, n_seg, L, Hq, Hkv, d, cap, n_ctx):
    g = torch.Generator().manual_seed(seed)
    q = torch.randn(n_seg, L, Hq, d, generator=g).to(torch.bfloat16).cuda()
    k = torch.randn(n_seg, cap, Hkv, d, generator=g).to(torch.bfloat16).cuda()
    v = torch.randn(n_seg, cap, Hkv, d, generator=g).to(torch.bfloat16).cuda()
    nc = torch.tensor(n_ctx, dtype=torch.int32).cuda()
    return q, k, v, nc


def both(q, k, v, nc, scale):
    """Output of the workspace entry point (NaN-filled workspace) and of the allocation-free
    one (NaN-filled output, so every element must be written)."""
    from paper_2609_34653_amd import omnitide as ot
    n_seg, L, Hq, d = q.shape
    cap, Hkv = k.shape[1], k.shape[2]
    nb = ot.omnitide_attn_workspace_bytes(n_seg, cap, L, Hq, Hkv, d)
    ws = torch.full((max(nb, 1) // 4 + 1,), float("nan"), device="cuda").view(torch.uint8)[:nb]
    ws = ws if nb else None
    ref = torch.full(q.shape, float("nan"), dtype=torch.float32, device="cuda")
    got = torch.full(q.shape, float("nan"), dtype=torch.float32, device="cuda")
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    ot.omnitide_chunk_attn(q, k, v, nc, scale, ref, ws, st)
    ot.omnitide_chunk_attn_noalloc(q, k, v, nc, scale, got, st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    return ref, got, nb


def test_noalloc_matches_workspace_entry_on_successive_calls():
    from paper_2609_34653_amd import omnitide as ot
    shapes = [
        # the 80K-history call: 665 queries, 32/8 heads, d 128 over 16,383 kept rows + the chunk
        (1, 1, 665, 32, 8, 128, 17100, [17048]),
        # smaller: two segments of the 1.6K workload's shape (89 queries, 4/1 heads, d 64)
        (2, 2, 89, 4, 1, 64, 601, [601, 400]),
        # one query over one tile: a single split, no scratch used
        (3, 1, 1, 8, 8, 128, 64, [40]),
    ]
    used = []
    for seed, n_seg, L, Hq, Hkv, d, cap, n_ctx in shapes:
        q, k, v, nc = inputs(seed, n_seg, L, Hq, Hkv, d, cap, n_ctx)
        ref, got, nb = both(q, k, v, nc, 1.0 / np.sqrt(d))
        assert nb <= ot.NOALLOC_SCRATCH_BYTES
        assert torch.isfinite(ref).all()
        assert torch.equal(got, ref), (n_seg, L, Hq, Hkv, d)
        used.append(nb)
    assert used[0] > used[1] > 0 and used[2] == 0   # sizes shrink; the last needs no scratch
