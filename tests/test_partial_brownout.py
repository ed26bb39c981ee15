"""Partial brownout: hot experts keep their own FFN, cold experts' calls go to
their united expert.

The oracle's segment map (``oracle/partial.py``) is pinned against what the
paper fixes about the threshold (the three brownout modes of Sec. 2.2; Sec. 5:
threshold 1 is zero brownout, 0 is full brownout) and against brute force
over every prefix of the frequency order; the library's host-side builder
(``paper_2607_04164_amd/brownout.py``) is checked against the oracle's; the
oracle layer over a segment map is checked against per-slot calls computed
with library matmuls (hot experts on their original weights, cold ones on the
united weights of Eq. 2).
"""
import numpy as np
import pytest
from scipy.special import expit

import oracle
from oracle.partial import hot_mask, partial_map
from paper_2607_04164_amd import brownout as BO
from paper_2607_04164_amd import workload as W


def _swiglu(x, wg, wu, wd):
    x = np.asarray(x, np.float64)
    g = x @ np.asarray(wg, np.float64).T
    u = x @ np.asarray(wu, np.float64).T
    return (g * expit(g) * u) @ np.asarray(wd, np.float64).T


def _rand_case(seed, E=12, G=4):
    r = np.random.default_rng(500 + seed)
    freq = r.dirichlet(np.full(E, 0.5))
    e2g = W.balanced_map(r.permutation(E), E, G)
    return freq, e2g


def test_theta_one_is_zero_brownout():
    freq, e2g = _rand_case(0)
    e2s, seg = partial_map(freq, e2g, 4, 1.0)
    assert np.array_equal(e2s, np.arange(12)), "every expert on its own FFN, in index order"
    assert seg == [("expert", e) for e in range(12)]


def test_theta_zero_is_full_brownout():
    freq, e2g = _rand_case(1)
    e2s, seg = partial_map(freq, e2g, 4, 0.0)
    assert np.array_equal(e2s, e2g), "every call goes to its united expert"
    assert seg == [("united", g) for g in range(4)]


def _hot_by_prefixes(freq, theta):
    """Brute force: the longest prefix of the order (frequency down, index up)
    whose total is within theta."""
    w = np.asarray(freq, np.float64) / np.sum(freq)
    order = np.lexsort((np.arange(len(w)), -w))
    best = 0
    for n in range(len(w) + 1):
        if w[order[:n]].sum() <= theta + 1e-9:
            best = n
    hot = np.zeros(len(w), bool)
    hot[order[:best]] = True
    return hot


@pytest.mark.parametrize("seed", range(6))
def test_hot_set_is_longest_prefix_within_theta(seed):
    freq, _ = _rand_case(seed, E=7)
    for theta in np.linspace(0, 1, 23):
        assert np.array_equal(hot_mask(freq, theta), _hot_by_prefixes(freq, theta)), theta


def test_hot_set_grows_with_theta_and_stays_within_it():
    freq, _ = _rand_case(7, E=20)
    w = freq / freq.sum()
    prev = np.zeros(20, bool)
    for theta in np.linspace(0, 1, 41):
        hot = hot_mask(freq, theta)
        assert np.all(hot[prev]), "monotone in theta"
        assert w[hot].sum() <= theta + 1e-9
        if not hot.all():  # maximal: the next expert of the order would exceed theta
            nxt = min(np.flatnonzero(~hot), key=lambda e: (-w[e], e))
            assert w[hot].sum() + w[nxt] > theta + 1e-9
        prev = hot


def test_ties_keep_the_lower_index():
    freq = np.array([0.2, 0.3, 0.2, 0.3])  # experts 1 and 3, then 0 and 2, tie pairwise
    assert hot_mask(freq, 0.3).tolist() == [False, True, False, False]
    assert hot_mask(freq, 0.8).tolist() == [True, True, False, True]


def test_segments_cover_the_map():
    freq, e2g = _rand_case(9, E=16, G=5)
    for theta in (0.2, 0.5, 0.8):
        e2s, seg = partial_map(freq, e2g, 5, theta)
        hot = hot_mask(freq, theta)
        assert len(seg) <= 16
        for e in range(16):
            kind, i = seg[e2s[e]]
            assert (kind, i) == (("expert", e) if hot[e] else ("united", int(e2g[e])))
        assert all(any(e2s[e] == s for e in range(16)) for s in range(len(seg))), "no unused segment"


@pytest.mark.parametrize("seed", range(5))
def test_library_builder_matches_oracle(seed):
    freq, e2g = _rand_case(seed, E=30, G=6)
    for theta in (0.0, 0.1, 0.37, 0.5, 0.9, 1.0):
        a = BO.segment_map(freq, e2g, 6, theta)
        b = partial_map(freq, e2g, 6, theta)
        assert np.array_equal(a[0], b[0]) and a[1] == b[1], theta


def test_library_builder_rejects_bad_input():
    """Host-side checks of the C call: nothing is built from a bad map, an
    out-of-range threshold or frequencies that are negative, non-finite or all
    zero."""
    freq, e2g = _rand_case(0)
    for theta in (-0.1, 1.5, float("nan")):
        with pytest.raises(ValueError):
            BO.segment_map(freq, e2g, 4, theta)
    bad = e2g.copy()
    bad[3] = 4
    with pytest.raises(ValueError):
        BO.segment_map(freq, bad, 4, 0.5)
    for f in (np.zeros(12), np.where(np.arange(12) == 2, -1.0, freq), np.where(np.arange(12) == 2, np.inf, freq)):
        with pytest.raises(ValueError):
            BO.segment_map(f, e2g, 4, 0.5)
    with pytest.raises(ValueError):
        BO.segment_map(freq, e2g, 13, 0.5)  # more groups than experts


def test_library_builder_ties_and_extremes():
    """Equal frequencies go to the lower index first; theta 0 and 1 give the
    group map and the identity."""
    freq = np.array([0.2, 0.1, 0.2, 0.1, 0.2, 0.2])
    e2g = np.array([0, 0, 1, 1, 2, 2], np.int32)
    e2s, seg = BO.segment_map(freq, e2g, 3, 0.45)
    assert seg[:2] == [("expert", 0), ("expert", 2)] and len(seg) == 2 + 3
    assert (e2s, seg) == (e2s, seg) and np.array_equal(*[partial_map(freq, e2g, 3, 0.45)[0], e2s])
    assert np.array_equal(BO.segment_map(freq, e2g, 3, 0.0)[0], e2g)
    assert np.array_equal(BO.segment_map(freq, e2g, 3, 1.0)[0], np.arange(6))


def test_partial_layer_is_per_slot_original_or_united_calls():
    cfg = W.LayerConfig("pb", T=24, d=32, E=10, top_k=3, G=3, d_ff=40, dtype="f32", zipf_s=1.0,
                        router_std=0.5, theta=0.5)
    L = W.make_layer(cfg, 3)
    freq = W.zipf_freq(L)
    e2s, seg = partial_map(freq, L.e2g, cfg.G, cfg.theta)
    hot = hot_mask(freq, cfg.theta)
    assert 0 < hot.sum() < cfg.E, "the case must mix original and united calls"
    PL = W.segment_layer(L, e2s, seg)
    res = oracle.layer(PL, want_intermediates=True)
    x = L.f32("x").astype(np.float64)
    ref = np.zeros((cfg.T, cfg.d))
    for t in range(cfg.T):
        for i in range(cfg.top_k):
            e = int(res["topk_idx"][t, i])
            w = W.expert_weights(L, e) if hot[e] else (L.w_gate[L.e2g[e]], L.w_up[L.e2g[e]], L.w_down[L.e2g[e]])
            ref[t] += float(res["topk_w"][t, i]) * _swiglu(x[t:t + 1], *w)[0]
    den = np.maximum(np.abs(ref).max(axis=1, keepdims=True), 1e-30)
    assert float((np.abs(res["out"] - ref) / den).max()) < 1e-5


def test_partial_workload_at_the_paper_threshold():
    """The bench workload: the fine-grained layer at threshold 0.4."""
    cfg = W.CONFIGS["partial"]
    assert cfg.theta == 0.4 and (cfg.E, cfg.top_k, cfg.G) == (60, 4, 15)
    L = W.make_layer(cfg.with_(T=8, d=64, d_ff=32), 0)
    e2s, seg = BO.segment_map(W.zipf_freq(L), L.e2g, cfg.G, cfg.theta)
    hot = [i for kind, i in seg if kind == "expert"]
    assert hot and len(seg) == len(hot) + cfg.G
    assert W.zipf_freq(L)[hot].sum() <= 0.4 + 1e-9
