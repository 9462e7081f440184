"""The whole stream step captured in one HIP graph: every replay, with eagerly launched steps and
synchronisations in between, reproduces the eagerly launched step bit for bit (the step issues
no memset nodes; accumulators are cleared by a kernel)."""
import numpy as np
import pytest
import torch

import streamgen as sg
from tests.test_gpu_parity import gpu_inputs, make_step, run_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_34653_amd import omnitide
    omnitide.lib()
    yield


@pytest.mark.parametrize("cfg_name", ["single_layer_8k", "history_80k"])
def test_step_graph_replays_match_eager(cfg_name):
    cfg = sg.CONFIG_BY_NAME[cfg_name]
    stream = sg.make_stream(cfg)
    lay, seg = stream.layout, stream.segment(0)
    st = make_step(cfg, lay)
    inp = gpu_inputs(lay, [seg])
    run_gpu(cfg, st, inp)
    ref = {k: getattr(st, k).clone() for k in ("out", "keep", "n_ctx", "k_dst", "v_dst",
                                               "unit_id_dst", "pos_dst", "unit_wsum")}
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run_gpu(cfg, st, inp, sync=False)
    for rep in range(4):
        for t in ref:                                    # poison the outputs
            getattr(st, t).zero_()
        g.replay()
        torch.cuda.synchronize()
        for t, want in ref.items():
            assert torch.equal(getattr(st, t), want), (rep, t)
        run_gpu(cfg, st, inp)                            # eager work between replays
        assert torch.equal(st.out, ref["out"])
    assert int(st.d_status.item()) == 0
