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
The map is built by the library's host-only call bmoe_partial_segment_map;
this module marshals numpy arrays into it and stacks the segments' weights.
"""
from __future__ import annotations

import ctypes
from typing import List, Tuple

import numpy as np

__all__ = ["hot_set", "segment_map", "stack_segments"]

_KIND = {0: "expert", 1: "united"}


def _build(freq, e2g, G: int, theta: float):
    from . import binding as B
    w = np.ascontiguousarray(freq, dtype=np.float64)
    m = np.ascontiguousarray(e2g, dtype=np.int32)
    if w.ndim != 1 or m.shape != w.shape:
        raise ValueError("freq and e2g must be 1-D arrays of the same length")
    E = w.shape[0]
    e2s = np.empty(E, np.int32)
    kind = np.empty(E, np.int32)
    sid = np.empty(E, np.int32)
    n = ctypes.c_int32(0)
    p = lambda a: a.ctypes.data_as(ctypes.c_void_p)  # noqa: E731
    st = B.load_library().bmoe_partial_segment_map(p(w), p(m), E, int(G), float(theta), p(e2s), p(kind), p(sid),
                                                   ctypes.byref(n))
    if st != 0:
        raise ValueError(f"bmoe_partial_segment_map: {B.status_str(st)}")
    return e2s, [(_KIND[int(kind[s])], int(sid[s])) for s in range(n.value)]


def hot_set(freq: np.ndarray, theta: float) -> np.ndarray:
    """Experts kept on their own FFN, ascending index."""
    w = np.asarray(freq, dtype=np.float64)
    _, segments = _build(w, np.zeros(w.shape[0], np.int32), 1, theta)
    return np.array([i for kind, i in segments if kind == "expert"], dtype=np.int32)


def segment_map(freq: np.ndarray, e2g: np.ndarray, G: int, theta: float) -> Tuple[np.ndarray, List[Tuple[str, int]]]:
    """Returns (e2s, segments): e2s[e] is the segment of expert e; segments[s]
    is ("expert", e) for a hot expert's own FFN or ("united", g) for a united
    expert."""
    return _build(freq, e2g, G, theta)


def stack_segments(segments, expert_w, united_w):
    """Weights of the segments in order: expert_w(e) and united_w(g) each
    return one FFN as (w_gate [d_ff, d], w_up [d_ff, d], w_down [d, d_ff])."""
    parts = [expert_w(i) if kind == "expert" else united_w(i) for kind, i in segments]
    return tuple(np.stack([p[j] for p in parts]) for j in range(3))
