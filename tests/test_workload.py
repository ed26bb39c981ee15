"""The seeded input generator (no GPU)."""
import math

import numpy as np
import pytest
from scipy.special import softmax

from paper_2607_04164_amd import workload as W


def test_same_seed_same_bytes():
    cfg = W.scaled(W.CONFIGS["fine"], T=40, d=64, d_ff=32)
    a, b = W.make_layer(cfg, 3), W.make_layer(cfg, 3)
    for name in ("e2g", "bias", "x", "w_router", "w_gate", "w_up", "w_down"):
        assert np.array_equal(getattr(a, name), getattr(b, name)), name
    c = W.make_layer(cfg, 4)
    assert not np.array_equal(a.x, c.x)


def test_bf16_rounding_is_rne():
    torch = pytest.importorskip("torch")
    r = np.random.default_rng(0)
    v = np.concatenate([r.standard_normal(10000).astype(np.float32) * 10.0 ** r.integers(-8, 8, 10000),
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.005859375, 3.4e38, -3.4e38, 1e-40],
                                 np.float32)]).astype(np.float32)
    ref = torch.from_numpy(v).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(W.f32_to_bf16_bits(v), ref)
    assert np.array_equal(W.bf16_bits_to_f32(ref), torch.from_numpy(ref.view(np.int16)).view(
        torch.bfloat16).float().numpy())


@pytest.mark.parametrize("name", ["tiny", "mixtral", "fine", "heavy", "decode"])
def test_map_and_bias_recipe(name):
    cfg = W.CONFIGS[name]
    L = W.make_layer(cfg, 0, with_weights=False)
    sizes = np.bincount(L.e2g, minlength=cfg.G)
    assert len(sizes) == cfg.G and sizes.min() >= 1 and sizes.max() <= math.ceil(cfg.E / cfg.G)
    # softmax of the bias is a Zipf(s) law over a permutation of ranks 1..E
    q = np.sort(softmax(L.bias.astype(np.float64)))[::-1]
    ranks = np.arange(1, cfg.E + 1, dtype=np.float64) ** -cfg.zipf_s
    assert np.allclose(q, ranks / ranks.sum(), rtol=1e-5)
    assert L.x.shape == (cfg.T, cfg.d)
    assert L.x.dtype == (np.float32 if cfg.dtype == "f32" else np.uint16)


def test_value_distributions():
    cfg = W.scaled(W.CONFIGS["heavy"], T=512, d=256, d_ff=64, E=16, G=4)
    L = W.make_layer(cfg, 1)
    x = L.f32("x")
    assert abs(x.std() - 1.0) < 0.02
    assert abs(L.f32("w_gate").std() - 1 / math.sqrt(cfg.d)) < 0.01 / math.sqrt(cfg.d) * 10
    assert L.w_gate_sh.shape == (1, cfg.d_ff_shared, cfg.d)
    assert L.w_down_sh.shape == (1, cfg.d, cfg.d_ff_shared)


def test_sequential_map_is_index_order():
    assert W.sequential_map(6, 2).tolist() == [0, 0, 1, 1, 2, 2]
    assert W.sequential_map(60, 4).max() == 14


def test_routed_load_is_as_skewed_as_the_paper_reports():
    """Sec. 2.3 (challenge C1): on the paper's 60-expert model the ten most
    used experts take more than 40 % of the routed tokens and the twenty least
    used fewer than 10 %. The synthetic skew of the 60-expert workload must be
    at least that strong (top-k picks on float64 logits of 2048 of its tokens)."""
    cfg = W.CONFIGS["fine"]
    L = W.make_layer(cfg, 0, with_weights=False)
    n = 2048
    z = L.f32("x")[:n].astype(np.float64) @ L.f32("w_router").astype(np.float64).T + L.bias
    picks = np.argsort(-z, axis=1, kind="stable")[:, :cfg.top_k]
    load = np.sort(np.bincount(picks.ravel(), minlength=cfg.E))[::-1] / picks.size
    assert load[:10].sum() > 0.40, load[:10].sum()
    assert load[-20:].sum() < 0.10, load[-20:].sum()
