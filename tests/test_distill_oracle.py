"""Pins of the grouping-search oracle (``oracle/distill.py``): the
distillation target of Eq. 5, the routing-weighted total of Eq. 6 and the
parameter-average initialisation of the united experts, against closed forms
and invariants the paper's definitions fix, plus planted mistakes that each
pin catches."""
import numpy as np
import pytest

import oracle
from oracle import distill as D


def _case(seed, E=7, G=3, T=5, d=4):
    r = np.random.default_rng(900 + seed)
    e2g = np.array([i % G for i in r.permutation(E)], dtype=np.int32)
    w = r.dirichlet(np.ones(E))
    y = r.standard_normal((E, T, d))
    return e2g, w, y


def test_alphas_normalise_frequencies_within_each_group():
    e2g, w, _ = _case(0)
    a = D.alphas(w, e2g, 3)
    for ms in D.members(e2g, 3):
        assert abs(sum(a[e] for e in ms) - 1.0) < 1e-15
        for e in ms:  # proportional to the frequency
            assert abs(a[e] * sum(w[f] for f in ms) - w[e]) < 1e-15


def test_group_with_zero_frequency_weighs_members_equally():
    a = D.alphas([0.0, 0.0, 0.5, 0.5], [0, 0, 1, 1], 2)
    assert a.tolist() == [0.5, 0.5, 0.5, 0.5]


def test_single_member_target_is_that_expert():
    e2g = np.array([0, 1, 1, 2], dtype=np.int32)
    _, w, y = _case(1, E=4)
    t = D.targets(y, w, e2g, 3)
    assert np.array_equal(t[0], y[0]) and np.array_equal(t[2], y[3])


def test_two_member_closed_form():
    """Members with constant outputs a and b, frequencies w1 and w2, united
    output 0: the target is (w1 a + w2 b) / (w1 + w2), the error its square."""
    a, b, w1, w2 = 3.0, 1.0, 0.2, 0.6
    y = np.stack([np.full((2, 3), a), np.full((2, 3), b)])
    mse, total = D.group_mse(np.zeros((1, 2, 3)), y, [w1, w2], [0, 0], 1)
    want = ((w1 * a + w2 * b) / (w1 + w2)) ** 2
    assert abs(mse[0] - want) < 1e-12 and abs(total - (w1 + w2) * want) < 1e-12


def test_constant_offset_gives_its_square_and_beta_weighting():
    e2g, w, y = _case(2)
    t = D.targets(y, w, e2g, 3)
    c = np.array([0.5, -2.0, 0.25])
    mse, total = D.group_mse(t + c[:, None, None], y, w, e2g, 3)
    assert np.allclose(mse, c ** 2, rtol=1e-12, atol=0)
    beta = np.array([w[e2g == r].sum() for r in range(3)])  # Eq. 6, written out here
    assert abs(total - float(np.dot(beta, c ** 2))) < 1e-12


def test_invariances():
    """Relabelling experts changes nothing; scaling the frequencies scales
    only the total; an empty group contributes nothing."""
    e2g, w, y = _case(3)
    u = np.random.default_rng(3).standard_normal((3,) + y.shape[1:])
    mse, total = D.group_mse(u, y, w, e2g, 3)
    p = np.random.default_rng(4).permutation(7)
    mse_p, total_p = D.group_mse(u, y[p], w[p], e2g[p], 3)
    assert np.allclose(mse_p, mse, rtol=1e-13) and abs(total_p - total) < 1e-12
    mse_s, total_s = D.group_mse(u, y, 5.0 * w, e2g, 3)
    assert np.allclose(mse_s, mse, rtol=1e-13) and abs(total_s - 5.0 * total) < 1e-11
    mse_e, total_e = D.group_mse(np.concatenate([u, u[:1]]), y, w, e2g, 4)
    assert mse_e[3] == 0.0 and abs(total_e - total) < 1e-15


def test_united_init_is_the_member_average():
    A, B, C = (np.random.default_rng(s).standard_normal((3, 2)) for s in (5, 6, 7))
    w = np.stack([A, B, C])
    init = D.united_init(w, [1, 0, 1], 2)
    assert np.array_equal(init[0], B)
    assert np.allclose(init[1], (A + C) / 2, rtol=0, atol=1e-15)
    assert np.array_equal(D.united_init(w[[2, 1, 0]], [1, 0, 1], 2), init)  # member order does not matter


def test_identical_members_distil_with_zero_error():
    """When a group's members share one FFN, their parameter average is that
    FFN, so the united expert reproduces the target exactly (Eq. 5 with any
    frequencies): MSE 0. Outputs from the layer oracle's FFN."""
    r = np.random.default_rng(8)
    d, f, T = 16, 24, 6
    x = r.standard_normal((T, d)).astype(np.float32)
    base = [r.standard_normal((f, d)).astype(np.float32), r.standard_normal((f, d)).astype(np.float32),
            r.standard_normal((d, f)).astype(np.float32)]
    E, G = 3, 1
    wg, wu, wd = (np.stack([m] * E) for m in base)
    ui = [D.united_init(m, [0] * E, G).astype(np.float32) for m in (wg, wu, wd)]
    offs = np.array([0, T], np.int32)
    y_e = np.stack([oracle.ffn(offs, x, wg[e:e + 1], wu[e:e + 1], wd[e:e + 1]) for e in range(E)])
    y_u = oracle.ffn(offs, x, *ui)[None]
    mse, total = D.group_mse(y_u, y_e, [0.1, 0.7, 0.2], [0] * E, G)
    # zero up to the rounding of the weighted sum 0.1 y + 0.7 y + 0.2 y
    assert mse[0] < 1e-28 * np.mean(y_e[0].astype(np.float64) ** 2) and total < 1e-28 * np.mean(y_e[0] ** 2)


# planted mistakes: each must fail one of the pins above

def _uniform_alphas(w_freq, e2g, G):
    a = np.zeros(len(w_freq))
    for ms in D.members(e2g, G):
        for e in ms:
            a[e] = 1.0 / len(ms)
    return a


def _unnormalised_alphas(w_freq, e2g, G):
    return np.asarray(w_freq, dtype=np.float64).copy()


@pytest.mark.parametrize("mutant", [_uniform_alphas, _unnormalised_alphas])
def test_mutant_alphas_are_caught(mutant, monkeypatch):
    monkeypatch.setattr(D, "alphas", mutant)
    with pytest.raises(AssertionError):
        test_two_member_closed_form()


def test_mutant_unweighted_total_is_caught(monkeypatch):
    monkeypatch.setattr(D, "betas", lambda w, e2g, G: np.ones(G))
    with pytest.raises(AssertionError):
        test_constant_offset_gives_its_square_and_beta_weighting()


def test_mutant_error_summed_over_features_is_caught(monkeypatch):
    real = D.group_mse

    def summed(u, y, w, e2g, G):
        mse, _ = real(u, y, w, e2g, G)
        mse = mse * np.asarray(u).shape[-1]
        return mse, float(np.dot(D.betas(w, e2g, G), mse))
    monkeypatch.setattr(D, "group_mse", summed)
    with pytest.raises(AssertionError):
        test_constant_offset_gives_its_square_and_beta_weighting()
