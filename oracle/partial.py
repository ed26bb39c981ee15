"""Partial-brownout segment map, oracle side.

TEST INFRASTRUCTURE ONLY (like the rest of this package); it shares no code
with the library's host-side map builder.

Definition (the brownout modes of Sec. 2.2 with the thresholds of Sec. 5:
threshold 1.0 keeps every original expert, 0 substitutes every call; the
paper does not define "cold" further, so this is the reading used): order
the experts by decreasing calibration frequency, ties by increasing index.
Expert e is hot exactly when the normalised frequency of the experts up to
and including e in that order is at most theta (1e-9 slack so that theta 1
keeps all). Hot experts keep their own FFN; every other expert's calls go to
its united expert g(e) (Eq. 2). Segments: the hot experts in increasing
index, then the united experts with at least one cold member in increasing
group index.
"""
from __future__ import annotations

import numpy as np

SLACK = 1e-9


def hot_mask(freq, theta: float) -> np.ndarray:
    """Boolean [E]: which experts stay on their own FFN (pairwise definition, O(E^2))."""
    w = np.asarray(freq, dtype=np.float64)
    w = w / w.sum()
    E = w.shape[0]
    hot = np.zeros(E, dtype=bool)
    for e in range(E):
        mass = 0.0
        for f in range(E):
            if w[f] > w[e] or (w[f] == w[e] and f <= e):
                mass += w[f]
        hot[e] = mass <= theta + SLACK
    return hot


def partial_map(freq, e2g, G: int, theta: float):
    """Returns (e2s [E] int32, segments: list of ("expert", e) / ("united", g))."""
    e2g = np.asarray(e2g, dtype=np.int32)
    hot = hot_mask(freq, theta)
    E = e2g.shape[0]
    segments = [("expert", e) for e in range(E) if hot[e]]
    groups = [g for g in range(G) if any((not hot[e]) and e2g[e] == g for e in range(E))]
    segments += [("united", g) for g in groups]
    index = {seg: s for s, seg in enumerate(segments)}
    e2s = np.array([index[("expert", e)] if hot[e] else index[("united", int(e2g[e]))] for e in range(E)],
                   dtype=np.int32)
    return e2s, segments
