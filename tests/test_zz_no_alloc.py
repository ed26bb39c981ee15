"""The allocation-free dispatch entry point against the workspace one.

brownout_moe_dispatch_noalloc runs the dispatch kernels on the library's own
per-device workspace array; its outputs must be bit-identical to
brownout_moe_dispatch's on a caller-owned workspace, call after call on the
same array, including a second, smaller call that finds the first call's
contents there.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from gpu_util import desc_of, dev_tensor
from paper_2607_04164_amd import binding as B
from paper_2607_04164_amd import workload as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load_library()


def _slots(cfg, seed):
    L = W.make_layer(cfg, seed, with_weights=False)
    r = oracle.route(L.f32("x"), L.f32("w_router"), L.bias, L.e2g, cfg.top_k, cfg.norm_topk)
    return L, r["slot_group"]


def _same(a, b, N, copy_rows):
    for key in ("counts", "offsets", "slot_row"):
        assert torch.equal(a[key], b[key]), key
    assert torch.equal(a["perm_token"][:N], b["perm_token"][:N])
    if copy_rows:
        assert torch.equal(a["x_perm"][:N].view(torch.int16), b["x_perm"][:N].view(torch.int16))


@pytest.mark.parametrize("copy_rows", [True, False], ids=["rows", "index-only"])
def test_noalloc_dispatch_matches_workspace_dispatch(copy_rows):
    """Two calls in a row on the library's array, the second on a smaller
    input; each against the workspace entry point and the oracle."""
    big = W.CONFIGS["fine"].with_(name="fine-noalloc", T=5000, d=256)
    small = W.CONFIGS["decode"].with_(name="decode-noalloc", d=256)
    for cfg, seed in ((big, 0), (small, 1), (big, 2)):
        L, sg_np = _slots(cfg, seed)
        desc = desc_of(cfg)
        sg = torch.from_numpy(sg_np).cuda()
        x = dev_tensor(L.x, cfg.dtype)
        ws = B.new_dispatch_workspace(desc, "cuda")
        want = B.dispatch(desc, sg, x if copy_rows else None, ws, copy_rows=copy_rows)
        got = B.dispatch_noalloc(desc, sg, x if copy_rows else None, copy_rows=copy_rows)
        torch.cuda.synchronize()
        ref = oracle.dispatch(sg_np, cfg.G)
        N = ref["N"]
        assert np.array_equal(got["offsets"].cpu().numpy(), ref["offsets"])
        _same(got, want, N, copy_rows)


def test_noalloc_dispatch_rejects_oversized_shapes():
    """A shape whose look-back state does not fit the array is refused before
    anything runs; the outputs stay untouched."""
    cfg = W.LayerConfig("huge", T=140000, d=64, E=256, top_k=2, G=256, d_ff=64, dtype="bf16", zipf_s=1.0)
    desc = desc_of(cfg)
    assert B.workspace_bytes(desc, B.STAGE_DISPATCH) > B.DISPATCH_SCRATCH_BYTES
    sg = torch.full((cfg.T, cfg.top_k), -1, dtype=torch.int32, device="cuda")
    offs = torch.full((cfg.G + 1,), 7, dtype=torch.int32, device="cuda")
    with pytest.raises(B.BmoeError) as e:
        B.dispatch_noalloc(desc, sg, None, copy_rows=False, out={"offsets": offs})
    assert e.value.status == B.STATUS_CODES["BMOE_ERR_WORKSPACE"]
    torch.cuda.synchronize()
    assert bool((offs == 7).all())
