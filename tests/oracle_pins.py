"""Pins of the CPU oracle against things other than the oracle itself.

Each ``pin_*`` takes an ``oracle.Oracle`` and raises AssertionError when the
oracle disagrees with:
  * a library routine on a special case (numpy/BLAS matmul, scipy softmax and
    logistic sigmoid), e.g. the ungrouped layer of Sec. 2.1 under the identity
    map, or top-k mass times one dense SwiGLU when G = 1;
  * brute force on tiny inputs (best k-subset of the logits);
  * invariants the layer's definition fixes (group weights sum to the top-k
    mass, merged and per-slot united-expert calls agree by linearity, the
    stable counting sort, token-order invariance);
  * the worked grouping example of the paper (Sec. 2.2, Fig. 1(a)) and Eq. 1.
The same pins run against deliberately broken builds of the oracle in
``test_oracle_mutants.py``: every planted mistake must trip at least one.
"""
from __future__ import annotations

import itertools
import json
import math
import os

import numpy as np
from scipy.special import expit, softmax

from paper_2607_04164_amd import workload as W

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _rng(seed):
    return np.random.default_rng(10_000 + seed)


def swiglu_lib(x, wg, wu, wd):
    """Dense SwiGLU with library primitives: silu(v) = v * logistic(v)."""
    x = np.asarray(x, np.float64)
    g = x @ np.asarray(wg, np.float64).T
    u = x @ np.asarray(wu, np.float64).T
    return (g * expit(g) * u) @ np.asarray(wd, np.float64).T


def _rand_layer(seed, T, d, E, k, G, d_ff, e2g=None, zipf=1.2, norm=0, n_shared=0):
    cfg = W.LayerConfig("pin", T=T, d=d, E=E, top_k=k, G=G, d_ff=d_ff, dtype="f32",
                        zipf_s=zipf, router_std=0.5, norm_topk=norm, n_shared=n_shared,
                        d_ff_shared_each=d_ff if n_shared else 0)
    L = W.make_layer(cfg, seed)
    if e2g is not None:
        L.e2g = np.asarray(e2g, np.int32)
    return L


def _topk_lib(z, k):
    """Reference selection: stable argsort of -z (ties -> lower index)."""
    return np.argsort(-z, kind="stable")[:k]


def _rel_rowmax(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    den = np.maximum(np.abs(b).max(axis=-1, keepdims=True), 1e-30)
    return float((np.abs(a - b) / den).max()) if a.size else 0.0


# ----------------------------------------------------------------------------
# gate

def pin_logits_vs_blas(orc):
    r = _rng(0)
    T, d, E = 9, 40, 7
    x = r.standard_normal((T, d)).astype(np.float32)
    w = r.standard_normal((E, d)).astype(np.float32)
    b = r.standard_normal(E).astype(np.float32)
    z = orc.router_logits(x, w, b)
    ref = x.astype(np.float64) @ w.astype(np.float64).T + b.astype(np.float64)
    assert np.allclose(z, ref, rtol=1e-12, atol=1e-12), np.abs(z - ref).max()


def pin_topk_best_subset(orc):
    r = _rng(1)
    for E in (1, 2, 5, 8, 9):
        for k in sorted({kk for kk in (1, 2, 3, E) if kk <= E}):
            z = r.standard_normal((6, E))
            out = orc.route_from_logits(z, np.zeros(E, np.int32), k)
            for t in range(z.shape[0]):
                best = max(itertools.combinations(range(E), k), key=lambda s: sum(z[t, list(s)]))
                got = out["topk_idx"][t]
                assert sorted(got.tolist()) == sorted(best), (E, k, got, best)
                assert np.all(np.diff(z[t, got]) <= 0), "slots must be in descending logit order"


def pin_topk_ties_lower_index(orc):
    z = np.array([[1.0, 2.0, 2.0, 1.0, 2.0],
                  [0.0, 0.0, 0.0, 0.0, 0.0],
                  [3.0, 1.0, 3.0, 3.0, -1.0]])
    out = orc.route_from_logits(z, np.zeros(5, np.int32), 3)
    assert out["topk_idx"].tolist() == [[1, 2, 4], [0, 1, 2], [0, 2, 3]], out["topk_idx"]
    for t in range(3):
        assert out["topk_idx"][t].tolist() == _topk_lib(z[t], 3).tolist()


def pin_softmax_weights(orc):
    r = _rng(2)
    z = r.standard_normal((20, 11)) * 3
    for norm in (0, 1):
        out = orc.route_from_logits(z, np.zeros(11, np.int32), 4, norm_topk=norm)
        p = softmax(z, axis=1)
        for t in range(20):
            ref = p[t, _topk_lib(z[t], 4)]
            if norm:
                ref = ref / ref.sum()
            assert np.allclose(out["topk_w"][t], ref, rtol=2e-7, atol=0), (norm, out["topk_w"][t], ref)


def pin_route_f32_logits_exact_values(orc):
    """Selection on float32 logits uses those exact values: the same picks,
    weights and groups as a library selection (stable argsort, scipy softmax)
    on the logits widened to float64, including values that tie only in
    float32 and a transposed-looking layout (T != E)."""
    r = _rng(8)
    T, E, k, G = 13, 10, 3, 4
    z = (r.standard_normal((T, E)) * 2).astype(np.float32)
    # two pairs that are equal in float32 (exact ties), one pair one ulp apart
    z[2, 7] = z[2, 4]
    z[5, 1] = z[5, 9] = np.float32(3.0)
    z[8, 3] = np.nextafter(z[8, 6], np.float32(np.inf))
    e2g = W.balanced_map(r.permutation(E), E, G)
    for norm in (0, 1):
        out = orc.route_from_logits(z, e2g, k, norm_topk=norm)
        z64 = z.astype(np.float64)
        p = softmax(z64, axis=1)
        for t in range(T):
            sel = _topk_lib(z64[t], k)
            assert out["topk_idx"][t].tolist() == sel.tolist(), (t, out["topk_idx"][t], sel)
            ref_w = p[t, sel] / (p[t, sel].sum() if norm else 1.0)
            assert np.allclose(out["topk_w"][t], ref_w, rtol=2e-7, atol=0), (t, norm)
            groups = e2g[sel]
            for i in range(k):
                if groups[i] in groups[:i]:
                    assert out["slot_group"][t, i] == -1 and out["slot_gate"][t, i] == 0
                else:
                    assert out["slot_group"][t, i] == groups[i]
                    want = ref_w[groups == groups[i]].sum()
                    assert math.isclose(out["slot_gate"][t, i], want, rel_tol=1e-6), (t, i)
        # the float64 entry on the widened values decides identically
        o64 = orc.route_from_logits(z64, e2g, k, norm_topk=norm)
        for key in ("topk_idx", "slot_group", "topk_w", "slot_gate"):
            assert np.array_equal(out[key], o64[key]), key


# ----------------------------------------------------------------------------
# substitution by united experts, merge

def pin_group_gates_sum_to_topk_mass(orc):
    r = _rng(3)
    for E, G, k in ((8, 4, 2), (12, 3, 5), (16, 1, 4), (10, 10, 3), (64, 8, 6)):
        z = r.standard_normal((50, E)) * 2
        e2g = W.balanced_map(r.permutation(E), E, G)
        out = orc.route_from_logits(z, e2g, k)
        sg, gate, w, idx = out["slot_group"], out["slot_gate"], out["topk_w"], out["topk_idx"]
        mass = w.astype(np.float64).sum(1)
        assert np.allclose(gate.astype(np.float64).sum(1), mass, rtol=k * 2.0 ** -23, atol=0)
        for t in range(50):
            groups = e2g[idx[t]]
            valid = sg[t] >= 0
            assert valid.sum() == len(set(groups.tolist()))
            assert np.all(gate[t][~valid] == 0)
            # each valid slot names its own pick's group, and that group appears first there
            for i in np.nonzero(valid)[0]:
                assert sg[t, i] == groups[i] and groups[i] not in groups[:i]


def pin_fig1_worked_maps(orc):
    g = json.load(open(os.path.join(GOLDEN, "fig1_worked_maps.json")))
    for case in g["cases"]:
        z = np.array([case["logits"]], np.float64)
        for name, m in g["maps"].items():
            out = orc.route_from_logits(z, np.array(m, np.int32), case["top_k"])
            assert out["topk_idx"][0].tolist() == case["topk_idx"], (case["desc"], name)
            assert out["slot_group"][0].tolist() == case["slot_group"][name], (case["desc"], name)
            # merged weight of a group = sum of its members' softmax weights
            p = softmax(z[0])
            for i, grp in enumerate(out["slot_group"][0]):
                if grp >= 0:
                    members = [e for e in case["topk_idx"] if m[e] == grp]
                    assert math.isclose(out["slot_gate"][0][i], p[members].sum(), rel_tol=1e-6)


# ----------------------------------------------------------------------------
# dispatch

def _check_dispatch(sg, d, G):
    T, k = sg.shape
    valid = sg >= 0
    counts = np.bincount(sg[valid], minlength=G)
    assert d["counts"].tolist() == counts.tolist()
    assert d["offsets"].tolist() == [0] + np.cumsum(counts).tolist()
    N = int(valid.sum())
    assert d["N"] == N and len(d["perm_token"]) == N
    rows = d["slot_row"][valid]
    assert sorted(rows.tolist()) == list(range(N)), "slot_row must be a bijection onto [0, N)"
    assert np.all(d["slot_row"][~valid] == -1)
    tt, ii = np.nonzero(valid)
    assert np.all(d["perm_token"][d["slot_row"][tt, ii]] == tt)
    for r in range(G):
        seg = d["perm_token"][d["offsets"][r]:d["offsets"][r + 1]]
        assert np.all(np.diff(seg) > 0), "rows of a group must be in ascending token order"
        for t in seg:
            assert r in sg[t].tolist()


def pin_dispatch_counting_sort(orc):
    r = _rng(4)
    for T, E, G, k in ((1, 4, 2, 2), (37, 8, 4, 2), (100, 60, 15, 4), (64, 64, 8, 6), (50, 5, 5, 1)):
        z = r.standard_normal((T, E))
        e2g = W.balanced_map(r.permutation(E), E, G)
        sg = orc.route_from_logits(z, e2g, k)["slot_group"]
        d = orc.dispatch(sg, G)
        _check_dispatch(sg, d, G)
        if k == 1:
            assert d["N"] == T


def pin_gather_rows(orc):
    r = _rng(5)
    x = r.standard_normal((10, 16)).astype(np.float32)
    perm = np.array([3, 3, 0, 9, 5], np.int32)
    assert np.array_equal(orc.gather_rows(x, perm), x[perm])


# ----------------------------------------------------------------------------
# whole layer

def _oracle_out(orc, L):
    return orc.layer(L, want_intermediates=True)


def pin_identity_map_is_ungrouped_layer(orc):
    """G = E with the identity map reduces to the plain top-K MoE layer of Sec. 2.1."""
    for seed, (T, d, E, k, f, norm) in enumerate(((16, 24, 6, 2, 40, 0), (9, 16, 8, 3, 24, 1))):
        L = _rand_layer(seed, T, d, E, k, E, f, e2g=np.arange(E), norm=norm)
        res = _oracle_out(orc, L)
        assert np.array_equal(res["slot_group"], res["topk_idx"]), "no merges under the identity map"
        x = L.f32("x").astype(np.float64)
        z = x @ L.f32("w_router").astype(np.float64).T + L.bias.astype(np.float64)
        p = softmax(z, axis=1)
        ref = np.zeros((T, d))
        for t in range(T):
            sel = _topk_lib(z[t], k)
            gw = p[t, sel] / (p[t, sel].sum() if norm else 1.0)
            for e, gi in zip(sel, gw):
                ref[t] += gi * swiglu_lib(x[t:t + 1], L.w_gate[e], L.w_up[e], L.w_down[e])[0]
        assert _rel_rowmax(res["out"], ref) < 1e-5, _rel_rowmax(res["out"], ref)


def pin_single_group_is_dense_ffn(orc):
    """G = 1: every token makes one call with weight equal to its top-k mass."""
    L = _rand_layer(7, 12, 32, 6, 3, 1, 48, e2g=np.zeros(6))
    res = _oracle_out(orc, L)
    x = L.f32("x").astype(np.float64)
    z = x @ L.f32("w_router").astype(np.float64).T + L.bias.astype(np.float64)
    p = softmax(z, axis=1)
    mass = np.array([p[t, _topk_lib(z[t], 3)].sum() for t in range(12)])
    ref = mass[:, None] * swiglu_lib(x, L.w_gate[0], L.w_up[0], L.w_down[0])
    assert res["N"] == 12 and np.all(res["counts"] == [12])
    assert _rel_rowmax(res["out"], ref) < 1e-5


def pin_merged_equals_per_slot_calls(orc):
    """One call with summed weights == one call per chosen expert (linearity)."""
    for seed, (T, d, E, k, G, f) in enumerate(((20, 24, 8, 4, 2, 32), (15, 16, 12, 5, 3, 16))):
        L = _rand_layer(20 + seed, T, d, E, k, G, f)
        res = _oracle_out(orc, L)
        assert (res["slot_group"] < 0).any(), "case must exercise merging"
        x = L.f32("x").astype(np.float64)
        ref = np.zeros((T, d))
        for t in range(T):
            for i in range(k):
                g = L.e2g[res["topk_idx"][t, i]]
                ref[t] += float(res["topk_w"][t, i]) * swiglu_lib(
                    x[t:t + 1], L.w_gate[g], L.w_up[g], L.w_down[g])[0]
        assert _rel_rowmax(res["out"], ref) < 1e-5


def pin_ffn_hidden_activation(orc):
    """The FFN's hidden output h is silu(gate) * up of each row against its own
    segment's weights (library matmuls, silu(v) = v * logistic(v)), and the
    down projection of h gives y."""
    r = _rng(9)
    n_seg, d, d_ff = 3, 20, 28
    offsets = np.array([0, 4, 4, 11], np.int32)  # an empty middle segment
    a = r.standard_normal((11, d)).astype(np.float32)
    wg = (r.standard_normal((n_seg, d_ff, d)) / 4).astype(np.float32)
    wu = (r.standard_normal((n_seg, d_ff, d)) / 4).astype(np.float32)
    wd = (r.standard_normal((n_seg, d, d_ff)) / 4).astype(np.float32)
    y, h = orc.ffn(offsets, a, wg, wu, wd, want_h=True)
    for s in range(n_seg):
        rows = slice(offsets[s], offsets[s + 1])
        a64 = a[rows].astype(np.float64)
        g = a64 @ wg[s].astype(np.float64).T
        u = a64 @ wu[s].astype(np.float64).T
        h_ref = g * expit(g) * u
        assert np.allclose(h[rows], h_ref, rtol=1e-6, atol=1e-7), s
        assert _rel_rowmax(y[rows], h_ref @ wd[s].astype(np.float64).T) < 1e-6, s


def pin_shared_experts_always_on(orc):
    L = _rand_layer(30, 10, 16, 8, 2, 4, 24, n_shared=2)
    res = _oracle_out(orc, L)
    routed = orc.combine(res["slot_row"], res["slot_gate"], res["y"], None, d=16)
    x = L.f32("x").astype(np.float64)
    ref = routed + swiglu_lib(x, L.w_gate_sh[0], L.w_up_sh[0], L.w_down_sh[0])
    assert _rel_rowmax(res["out"], ref) < 1e-5


def pin_token_order_invariance(orc):
    L = _rand_layer(40, 33, 16, 12, 3, 4, 24)
    res = _oracle_out(orc, L)
    perm = _rng(6).permutation(33)
    L2 = _rand_layer(40, 33, 16, 12, 3, 4, 24)
    L2.x = L.x[perm].copy()
    res2 = _oracle_out(orc, L2)
    assert np.array_equal(res2["out"], res["out"][perm])
    assert np.array_equal(res2["counts"], res["counts"])
    assert np.array_equal(res2["slot_group"], res["slot_group"][perm])


def pin_eq1_group_counts(orc):
    g = json.load(open(os.path.join(GOLDEN, "eq1_group_counts.json")))
    E = g["E"]
    for kway, G in g["G_for_k_way"].items():
        assert math.ceil(E / int(kway)) == G
        cap = g["capacity_for_G"][str(G)]
        assert math.ceil(E / G) == cap
        m = W.balanced_map(np.arange(E)[::-1], E, G)
        sizes = np.bincount(m, minlength=G)
        assert sizes.min() >= 1 and sizes.max() <= cap
        # a balanced map routes through the oracle like any other map
        z = _rng(7).standard_normal((5, E))
        assert orc.route_from_logits(z, m, 4)["slot_group"].max() < G


ALL_PINS = [
    pin_logits_vs_blas, pin_topk_best_subset, pin_topk_ties_lower_index, pin_softmax_weights,
    pin_route_f32_logits_exact_values, pin_ffn_hidden_activation,
    pin_group_gates_sum_to_topk_mass, pin_fig1_worked_maps, pin_dispatch_counting_sort,
    pin_gather_rows, pin_identity_map_is_ungrouped_layer, pin_single_group_is_dense_ffn,
    pin_merged_equals_per_slot_calls, pin_shared_experts_always_on, pin_token_order_invariance,
    pin_eq1_group_counts,
]
