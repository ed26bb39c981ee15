"""The layer captured into a HIP graph (torch.cuda.CUDAGraph): every replay
equals the eager forward bit for bit, also after the input changes between
replays and with eager work in between; the dispatch workspace is left zero
after each replay (the library's calls clear their own state with kernels, no
memset nodes and no host synchronisation inside)."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from gpu_util import desc_of, dev_tensor, device_weights
from paper_2607_04164_amd import binding as B
from paper_2607_04164_amd import workload as W

pytestmark = pytest.mark.gpu

CASES = {
    # the persistent 256-row GEMM tiles with the stream-K split
    "mixtral-s": W.CONFIGS["mixtral"].with_(name="mixtral-s", T=2100, d=256, d_ff=384),
    # decode-sized: the skinny GEMMs and the one-kernel dispatch
    "decode": W.CONFIGS["decode"],
    # shared experts
    "heavy-s": W.CONFIGS["heavy"].with_(name="heavy-s", T=700, d=512, d_ff=192, d_ff_shared_each=192),
}


@pytest.fixture(scope="module", autouse=True)
def _lib():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load_library()


@pytest.mark.parametrize("name", list(CASES))
@pytest.mark.parametrize("fold", [False, True], ids=["four-calls", "fold-combine"])
def test_layer_graph_replay(name, fold):
    cfg = CASES[name]
    L0 = W.make_layer(cfg, 0)
    L1 = W.make_layer(cfg, 1, with_weights=False)  # a second input for the same weights
    layer = B.LayerForward(desc_of(cfg), device_weights(L0), fold_combine=fold)
    x = dev_tensor(L0.x, cfg.dtype)
    x0 = x.clone()
    x1 = dev_tensor(L1.x, cfg.dtype)
    eager0 = layer(x).clone()
    layer(x1)
    eager1 = layer.bufs["out"].clone()
    torch.cuda.synchronize()
    # warm up on a side stream, then capture one forward
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        layer(x)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        out = layer(x)
    for rep, (src, want) in enumerate([(x0, eager0), (x1, eager1), (x0, eager0), (x1, eager1)]):
        x.copy_(src)
        layer.bufs["out"].zero_()
        layer.bufs["y"].zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, want), f"replay {rep}"
        assert int(layer.ws.count_nonzero()) == 0, f"dispatch workspace after replay {rep}"
        if fold:
            assert int(layer.fold_ws.count_nonzero()) == 0, f"fold workspace after replay {rep}"
    # eager forwards still agree after the replays
    assert torch.equal(layer(x0).clone(), eager0)
    del g
    torch.cuda.synchronize()
    assert np.isfinite(eager0.float().cpu().numpy()).all()
