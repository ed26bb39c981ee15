"""Partial brownout: the segment map that keeps hot experts on their own FFN.

The brownout approach has three modes (Sec. 2.2): zero brownout keeps every
original expert, full brownout sends every call to the united expert of its
group, and partial brownout substitutes only the calls of cold experts,
chosen by a threshold (Sec. 5, baselines: threshold 1.0 is zero brownout, 0
is full brownout; Sec. 4.3, closing paragraph: the gate still picks the
experts and only eligible cold calls are replaced through the saved map;
Sec. 4.5: the serving controller moves the threshold).

Reading of the threshold (the paper does not define "cold" further): with
per-expert routing frequencies w (from calibration), the hot set is the
longest run of experts in order of decreasing w (ties: lower index first)
whose cumulative frequency does not exceed theta. Theta 1 keeps every expert,
theta 0 none.

The layer then runs unchanged over S segments: the hot experts (ascending
index) with their original weights, followed by the united experts that still
have a cold member (ascending group index) with their united weights; the
segment map e2s replaces e2g in route, dispatch, FFN and combine. S <= E.
This module is host-side numpy; the layer's arithmetic stays in the library.
"""
from __future__ import annotations

from typing import List, Tuple

import numpy as np

__all__ = ["hot_set", "segment_map", "stack_segments"]

# slack for the cumulative comparison, so that theta = 1 keeps every expert
# whatever the rounding of the frequency sum
_SLACK = 1e-9


def hot_set(freq: np.ndarray, theta: float) -> np.ndarray:
    """Experts kept on their own FFN, ascending index."""
    w = np.asarray(freq, dtype=np.float64)
    if w.ndim != 1 or np.any(w < 0) or not np.all(np.isfinite(w)):
        raise ValueError("freq must be a 1-D array of finite non-negative frequencies")
    if not 0.0 <= theta <= 1.0:
        raise ValueError("theta must lie in [0, 1]")
    tot = w.sum()
    if tot <= 0:
        raise ValueError("frequencies sum to zero")
    order = sorted(range(len(w)), key=lambda e: (-w[e], e))
    hot, acc = [], 0.0
    for e in order:
        if acc + w[e] / tot > theta + _SLACK:
            break
        acc += w[e] / tot
        hot.append(e)
    return np.array(sorted(hot), dtype=np.int32)


def segment_map(freq: np.ndarray, e2g: np.ndarray, G: int, theta: float) -> Tuple[np.ndarray, List[Tuple[str, int]]]:
    """Returns (e2s, segments): e2s[e] is the segment of expert e; segments[s]
    is ("expert", e) for a hot expert's own FFN or ("united", g) for a united
    expert."""
    e2g = np.asarray(e2g, dtype=np.int32)
    E = e2g.shape[0]
    if np.any(e2g < 0) or np.any(e2g >= G):
        raise ValueError("e2g must map into [0, G)")
    hot = hot_set(freq, theta)
    is_hot = np.zeros(E, dtype=bool)
    is_hot[hot] = True
    segments: List[Tuple[str, int]] = [("expert", int(e)) for e in hot]
    used = sorted({int(e2g[e]) for e in range(E) if not is_hot[e]})
    seg_of_group = {g: len(hot) + i for i, g in enumerate(used)}
    segments += [("united", g) for g in used]
    e2s = np.empty(E, dtype=np.int32)
    for e in range(E):
        e2s[e] = np.searchsorted(hot, e) if is_hot[e] else seg_of_group[int(e2g[e])]
    return e2s, segments


def stack_segments(segments, expert_w, united_w):
    """Weights of the segments in order: expert_w(e) and united_w(g) each
    return one FFN as (w_gate [d_ff, d], w_up [d_ff, d], w_down [d, d_ff])."""
    parts = [expert_w(i) if kind == "expert" else united_w(i) for kind, i in segments]
    return tuple(np.stack([p[j] for p in parts]) for j in range(3))
