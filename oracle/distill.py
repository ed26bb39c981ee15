"""Grouping-search quantities of one layer, oracle side: the distillation
target of each united expert and the routing-weighted total MSE.

TEST INFRASTRUCTURE ONLY (like the rest of this package); it shares no code
with the library's kernels. Plain numpy in float64, following the paper's
definitions in order:

  * united-expert initialisation: the parameter average of the member
    experts (Sec. 4.3, after Eq. 5);
  * distillation target (Eq. 5): alpha_e = w_e / sum of w over the group,
    t_k(x) = sum over the members e of alpha_e f_e(x);
  * group error and total (Eq. 3, Eq. 6): beta_r = sum of w over group r,
    MSE_total = sum over r of beta_r MSE_r.

Readings where the paper is silent: MSE_r is the mean over the calibration
tokens and the output dimensions of (f_u_r(x) - t_r(x))^2, every group
evaluated on the same calibration tokens; a group whose members have zero
total frequency weighs its members equally in the target; an empty group has
MSE 0 and beta 0.
"""
from __future__ import annotations

import numpy as np


def members(e2g, G: int):
    """Member experts of each group, ascending (entries outside [0, G) belong to none)."""
    e2g = np.asarray(e2g)
    return [[e for e in range(e2g.shape[0]) if e2g[e] == r] for r in range(G)]


def united_init(w_expert: np.ndarray, e2g, G: int) -> np.ndarray:
    """Parameter average of the members, float64: w_expert [E, ...] -> [G, ...]
    (zeros for an empty group)."""
    w = np.asarray(w_expert, dtype=np.float64)
    out = np.zeros((G,) + w.shape[1:], dtype=np.float64)
    for r, ms in enumerate(members(e2g, G)):
        if ms:
            out[r] = sum(w[e] for e in ms) / len(ms)
    return out


def alphas(w_freq, e2g, G: int) -> np.ndarray:
    """alpha_e of Eq. 5 (0 for an expert in no group)."""
    w = np.asarray(w_freq, dtype=np.float64)
    a = np.zeros(w.shape[0])
    for ms in members(e2g, G):
        if not ms:
            continue
        tot = sum(w[e] for e in ms)
        for e in ms:
            a[e] = w[e] / tot if tot > 0 else 1.0 / len(ms)
    return a


def betas(w_freq, e2g, G: int) -> np.ndarray:
    """beta_r of Eq. 6."""
    w = np.asarray(w_freq, dtype=np.float64)
    return np.array([sum(w[e] for e in ms) for ms in members(e2g, G)], dtype=np.float64)


def targets(y_expert: np.ndarray, w_freq, e2g, G: int) -> np.ndarray:
    """t_k(x) of Eq. 5 for every group: y_expert [E, T, d] -> [G, T, d]."""
    y = np.asarray(y_expert, dtype=np.float64)
    a = alphas(w_freq, e2g, G)
    t = np.zeros((G,) + y.shape[1:])
    for r, ms in enumerate(members(e2g, G)):
        for e in ms:
            t[r] += a[e] * y[e]
    return t


def group_mse(y_united: np.ndarray, y_expert: np.ndarray, w_freq, e2g, G: int):
    """(MSE_r for every group [G], MSE_total) from the united experts' outputs
    [G, T, d] and the member experts' outputs [E, T, d]."""
    u = np.asarray(y_united, dtype=np.float64)
    t = targets(y_expert, w_freq, e2g, G)
    mse = np.zeros(G)
    for r, ms in enumerate(members(e2g, G)):
        if ms:
            mse[r] = np.mean((u[r] - t[r]) ** 2)
    return mse, float(np.dot(betas(w_freq, e2g, G), mse))
