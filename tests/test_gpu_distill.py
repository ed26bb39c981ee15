"""Grouping-search kernels (united init, distillation error) against the
oracle of ``oracle/distill.py``, through the C ABI (needs an MI355X)."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from oracle import distill as D
from gpu_util import assert_close_rows, dev_tensor, host_f32, to_storage
from paper_2607_04164_amd import binding as B
from paper_2607_04164_amd import workload as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _lib():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load_library()


def _experts(cfg, seed):
    """Seeded original FFNs of every expert, stacked, storage format."""
    L = W.make_layer(cfg, seed, with_weights=False)
    parts = [W.expert_weights(L, e) for e in range(cfg.E)]
    return L, tuple(np.stack([p[j] for p in parts]) for j in range(3))


MAPS = {
    "balanced": None,                                         # the workload's map
    "empty+single": np.array([0, 0, 2, 2, 2, 3, 0, 3, 2, 0, 0, 2], dtype=np.int32),  # group 1 empty
}


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("mapname", list(MAPS))
def test_united_init(dtype, mapname):
    cfg = W.LayerConfig("ui", T=8, d=256, E=12, top_k=2, G=4, d_ff=384, dtype=dtype, zipf_s=1.0)
    L, (wg, wu, wd) = _experts(cfg, 2)
    e2g = L.e2g if MAPS[mapname] is None else MAPS[mapname]
    out = B.united_init(torch.from_numpy(e2g).cuda(), cfg.G, dev_tensor(wg, dtype), dev_tensor(wu, dtype),
                        dev_tensor(wd, dtype))
    torch.cuda.synchronize()
    for got, w in zip(out, (wg, wu, wd)):
        want = D.united_init(W.bf16_bits_to_f32(w) if dtype == "bf16" else w, e2g, cfg.G)
        g = host_f32(got).astype(np.float64)
        if dtype == "f32":
            assert np.array_equal(g, want.astype(np.float32).astype(np.float64))
        else:
            # one rounding to bf16 (the kernel's fp32 sum and division may round
            # once more): within one bf16 step of the float64 average
            step = np.maximum(np.abs(want), 2.0 ** -126) * 2.0 ** -7
            assert np.all(np.abs(g - want) <= step)
            assert np.mean(g == W.bf16_bits_to_f32(W.f32_to_bf16_bits(want.astype(np.float32)))) > 0.999
        if mapname != "balanced":
            assert not g[1].any(), "an empty group is zero"


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("T", [1, 300, 4099])
def test_distill_mse_on_given_outputs(dtype, T):
    """The error reduction alone, on outputs handed to both sides: float64
    oracle against fp32 targets and fp64 sums; a group with zero total
    frequency and an empty group included."""
    E, G, d = 12, 5, 264
    r = np.random.default_rng(T)
    e2g = np.array([0, 0, 2, 2, 2, 3, 0, 3, 2, 0, 0, 4], dtype=np.int32)  # group 1 empty
    w = r.dirichlet(np.ones(E)).astype(np.float32)
    w[[5, 7]] = 0.0  # group 3: zero total frequency
    y_e = to_storage(r.standard_normal((E * T, d)).astype(np.float32), dtype)
    y_u = to_storage(r.standard_normal((G * T, d)).astype(np.float32), dtype)
    mse, total = B.distill_mse(torch.from_numpy(e2g).cuda(), torch.from_numpy(w).cuda(), dev_tensor(y_e, dtype),
                               dev_tensor(y_u, dtype), T)
    torch.cuda.synchronize()
    f = (lambda a: W.bf16_bits_to_f32(a)) if dtype == "bf16" else (lambda a: a)
    want, want_total = D.group_mse(f(y_u).reshape(G, T, d), f(y_e).reshape(E, T, d), w.astype(np.float64), e2g, G)
    got = mse.cpu().numpy()
    assert got[1] == 0.0 and want[1] == 0.0
    assert np.allclose(got, want, rtol=2e-6, atol=0), (got, want)
    assert abs(float(total.item()) - want_total) <= 2e-6 * abs(want_total)
    mse2, total2 = B.distill_mse(torch.from_numpy(e2g).cuda(), torch.from_numpy(w).cuda(), dev_tensor(y_e, dtype),
                                 dev_tensor(y_u, dtype), T)
    torch.cuda.synchronize()
    assert torch.equal(mse2, mse) and torch.equal(total2, total), "deterministic"


@pytest.mark.parametrize("seed", [0, 1])
def test_grouping_evaluation_end_to_end(seed):
    """One candidate map evaluated the way the search does, all on the GPU:
    expert outputs on the calibration tokens (one gathered FFN segment per
    expert), parameter-average united experts, their outputs, then the
    errors, against the oracle's own chain (float64 averages, float64 FFN
    sums rounded to float, float64 errors)."""
    cfg = W.LayerConfig("gs", T=300, d=256, E=12, top_k=2, G=4, d_ff=384, dtype="bf16", zipf_s=1.0)
    L, (wg, wu, wd) = _experts(cfg, 10 + seed)
    T, E, G = cfg.T, cfg.E, cfg.G
    wfreq = W.zipf_freq(L).astype(np.float32)
    e2g_d = torch.from_numpy(L.e2g).cuda()
    x = dev_tensor(L.x, "bf16")
    we = [dev_tensor(m, "bf16") for m in (wg, wu, wd)]
    y_e = B.ffn_all_tokens(x, *we)
    wu_g = B.united_init(e2g_d, G, *we)
    y_u = B.ffn_all_tokens(x, *wu_g)
    mse, total = B.distill_mse(e2g_d, torch.from_numpy(wfreq).cuda(), y_e, y_u, T)
    torch.cuda.synchronize()

    xf = L.f32("x")
    offs = np.array([0, T], np.int32)
    f = [W.bf16_bits_to_f32(m) for m in (wg, wu, wd)]
    ye_o = np.stack([oracle.ffn(offs, xf, f[0][e:e + 1], f[1][e:e + 1], f[2][e:e + 1]) for e in range(E)])
    ui = [D.united_init(m, L.e2g, G).astype(np.float32) for m in f]
    yu_o = np.stack([oracle.ffn(offs, xf, ui[0][r:r + 1], ui[1][r:r + 1], ui[2][r:r + 1]) for r in range(G)])
    want, want_total = D.group_mse(yu_o, ye_o, wfreq.astype(np.float64), L.e2g, G)

    # intermediate outputs at the layer's bf16 tolerance
    assert_close_rows(host_f32(y_e), ye_o.reshape(E * T, -1), "bf16", "expert outputs")
    assert_close_rows(host_f32(y_u), yu_o.reshape(G * T, -1), "bf16", "united outputs")
    # errors: the GPU's outputs carry bf16 roundings (united weights, h, y),
    # each within 2^-8 relative; with e = 2^-6 the difference (u - t) moves
    # by at most about e * rms(t) per element, so |dMSE| <= 2 e sqrt(MSE) rms(t) + e^2 rms(t)^2
    t = D.targets(ye_o, wfreq.astype(np.float64), L.e2g, G)
    got = mse.cpu().numpy()
    e = 2.0 ** -6
    for r in range(G):
        rms = float(np.sqrt(np.mean(t[r] ** 2)))
        tol = 2 * e * np.sqrt(want[r]) * rms + (e * rms) ** 2
        assert abs(got[r] - want[r]) <= tol, (r, got[r], want[r], tol)
    assert want_total > 0 and abs(float(total.item()) - want_total) <= 0.05 * want_total
