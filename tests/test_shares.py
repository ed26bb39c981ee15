"""One GPU's share of a layer sharded over several GPUs (CPU checks).

Under tensor parallelism each rank holds a slice of every FFN's hidden
columns and produces a partial output; under expert parallelism each rank
runs the grouped FFN for its block of united experts. What the shares must
add up to follows from the layer's definition (Sec. 2.1: the output is a sum
over the picked experts of their FFN outputs, and an FFN's down projection is
a sum over its hidden columns), so the oracle's shares are pinned against the
oracle's whole layer.
"""
import numpy as np
import pytest

import oracle
from paper_2607_04164_amd import workload as W

CFG = W.LayerConfig("tps", T=40, d=32, E=8, top_k=2, G=4, d_ff=48, dtype="f32", zipf_s=1.0,
                    router_std=0.5, norm_topk=1, n_shared=2, d_ff_shared_each=24)


def _rows_rel(a, b):
    den = np.maximum(np.abs(b).max(axis=1, keepdims=True), 1e-30)
    return float((np.abs(a - b) / den).max())


@pytest.mark.parametrize("P", [1, 2, 3, 4, 8])
def test_tp_shares_add_up_to_the_layer(P):
    L = W.make_layer(CFG, 4)
    full = oracle.layer(L).astype(np.float64)
    parts = [oracle.layer(W.tp_share(L, P, r)).astype(np.float64) for r in range(P)]
    # every share routes identically; each partial output is rounded to float once
    assert _rows_rel(sum(parts), full) < 1e-5 * (P + 1)
    if P > 1:
        assert _rows_rel(parts[0], full) > 1e-2, "a share alone is not the layer"


def test_tp_share_of_one_rank_is_the_layer():
    L = W.make_layer(CFG, 5)
    S = W.tp_share(L, 1, 0)
    for k in ("w_gate", "w_up", "w_down", "w_gate_sh", "w_up_sh", "w_down_sh"):
        assert np.array_equal(getattr(S, k), getattr(L, k)), k
    assert S.cfg.d_ff == CFG.d_ff and S.cfg.d_ff_shared == CFG.d_ff_shared


def test_tp_share_slices_each_shared_expert():
    """The shared-expert slice takes columns of each shared expert, not a
    block of the concatenation: with 2 shared experts of 24 and P=4, rank 1
    holds columns 6..11 and 30..35."""
    L = W.make_layer(CFG, 6)
    S = W.tp_share(L, 4, 1)
    cols = np.r_[6:12, 30:36]
    assert np.array_equal(S.w_gate_sh[0], L.w_gate_sh[0][cols])
    assert np.array_equal(S.w_down_sh[0], L.w_down_sh[0][:, cols])
    assert np.array_equal(S.w_up[2], L.w_up[2][12:24])


def test_tp_share_rejects_uneven_splits():
    L = W.make_layer(CFG, 0)
    with pytest.raises(ValueError):
        W.tp_share(L, 5, 0)
    with pytest.raises(ValueError):
        W.tp_share(L, 4, 4)


@pytest.mark.parametrize("G,P", [(15, 4), (4, 4), (4, 8), (16, 16), (60, 7)])
def test_ep_groups_partition(G, P):
    blocks = [W.ep_groups(G, P, r) for r in range(P)]
    assert blocks[0][0] == 0 and blocks[-1][1] == G
    assert all(blocks[i][1] == blocks[i + 1][0] for i in range(P - 1))
    sizes = [b - a for a, b in blocks]
    assert max(sizes) - min(sizes) <= 1


def test_ep_shares_reproduce_the_ffn_rows():
    """The FFN over one rank's block, on the rows that rank receives (packed
    from row 0), gives the whole FFN's rows for that block, bit for bit."""
    L = W.make_layer(CFG.with_(T=64), 7)
    ref = oracle.layer(L, want_intermediates=True)
    offs = ref["offsets"]
    for r in range(3):
        g0, g1 = W.ep_groups(CFG.G, 3, r)
        lo, hi = offs[g0], offs[g1]
        y = oracle.ffn(offs[g0:g1 + 1] - lo, ref["x_perm"][lo:hi], L.w_gate[g0:g1], L.w_up[g0:g1],
                       L.w_down[g0:g1])
        assert np.array_equal(y, ref["y"][lo:hi]), r
