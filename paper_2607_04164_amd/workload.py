"""Seeded synthetic workloads for the grouped (full-brownout) MoE layer.

This module only draws inputs. It holds none of the layer's arithmetic: it
makes token activations, router weights, a per-expert skew bias, an
expert-to-group map and united-expert SwiGLU weights from a seed, and hands
the same bytes to every consumer (the HIP path and the CPU oracle).

Workload recipe (per layer configuration):

* Generator: ``numpy.random.default_rng(seed)`` (PCG64). Draw order is fixed:
  map permutation, Zipf rank permutation, x, W_router, then W_gate, W_up,
  W_down (all united experts at once, in that order), then the shared-expert
  weights if the configuration has any.
* ``N(0, s)`` means standard deviation ``s``. x ~ N(0, 1); W_router ~
  N(0, router_std) (``1/sqrt(d)`` unless the configuration fixes it); every
  FFN weight ~ N(0, 1/sqrt(d)).
* bf16 configurations round every tensor to bf16 once, round-to-nearest-even;
  both sides then consume those exact bytes (the oracle widens them to fp32,
  which is exact).
* Expert-to-group map (the map g of Eq.2, 0-based): with a seeded permutation
  pi of the E experts, expert pi[i] goes to group floor(i*G/E). Groups then
  hold floor(E/G) or ceil(E/G) experts, never more than the capacity
  ceil(E/G) of the grouping search (Sec. 4.3), and every group is non-empty
  when G <= E.
* Hot/cold skew: with a seeded rank permutation rho (values 1..E), expert e
  gets the additive router bias ln(q_e), q_e = rho_e^-s / sum rho^-s, so that
  softmax(bias) is a Zipf(s) law over randomly placed hot experts. This stands
  in for the long-tailed expert load the paper reports on its model
  (Sec. 2.3, challenge C1); the paper's model, traces and weights are not used.
* Shared experts (heavy-skew configuration): ``n_shared`` always-on SwiGLU
  experts of width ``d_ff_shared_each``; their gate/up rows and down columns
  are concatenated into one FFN of width n_shared*d_ff_shared_each, which is
  the same function as their sum.
* Partial brownout (configurations with a threshold ``theta``): the original
  FFN of expert e is drawn from its own generator,
  ``default_rng([seed, 1_000_000 + e])`` (gate, up, down; same distribution
  as the united experts), so any subset of experts can be drawn alone. The
  calibration frequencies that pick the hot experts stand in as the Zipf law
  of the skew bias (``zipf_freq``); the paper's calibration traces are not
  here. ``segment_layer`` assembles the layer over a segment map (hot
  experts' own FFNs, then united experts); the map itself comes from the
  caller.
* Shares of a multi-GPU layer on one GPU: ``tp_share`` is rank r's share
  under tensor parallelism over P GPUs (columns r*d_ff/P .. (r+1)*d_ff/P - 1
  of every united expert's hidden width, and the same slice of each shared
  expert; route and dispatch are replicated, and the P partial outputs add
  up to the layer's output); ``ep_groups`` is rank r's block of united
  experts under expert parallelism (contiguous, sizes differing by at most
  one). Both only select existing weights.
"""
from __future__ import annotations

import dataclasses
import math
import os
from typing import Dict, Optional

import numpy as np

__all__ = ["LayerConfig", "CONFIGS", "Layer", "make_layer", "bf16_round_bits",
           "bf16_bits_to_f32", "f32_to_bf16_bits", "scaled", "tp_share", "ep_groups"]


@dataclasses.dataclass(frozen=True)
class LayerConfig:
    """Shape and value distribution of one grouped MoE layer workload."""
    name: str
    T: int            # tokens in the batch
    d: int            # model width
    E: int            # routed experts before grouping
    top_k: int        # experts picked per token by the gate
    G: int            # united experts after grouping
    d_ff: int         # SwiGLU hidden width of each united expert
    dtype: str        # "f32" or "bf16"
    zipf_s: float     # Zipf exponent of the per-expert skew bias
    router_std: Optional[float] = None   # None -> 1/sqrt(d)
    norm_topk: int = 0                   # renormalise the top-k weights to sum 1
    n_shared: int = 0                    # always-on shared experts
    d_ff_shared_each: int = 0
    theta: Optional[float] = None        # partial-brownout threshold (None: full brownout)

    @property
    def d_ff_shared(self) -> int:
        return self.n_shared * self.d_ff_shared_each

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    def with_(self, **kw) -> "LayerConfig":
        return dataclasses.replace(self, **kw)


# The five workloads the layer is measured and tested on.
CONFIGS: Dict[str, LayerConfig] = {
    # tiny fp32 layer, small enough for every oracle check
    "tiny": LayerConfig("tiny", T=64, d=256, E=8, top_k=2, G=4, d_ff=512,
                        dtype="f32", zipf_s=1.2, router_std=0.02),
    # Mixtral-8x7B-shaped layer, 2 experts per united expert
    "mixtral": LayerConfig("mixtral", T=4096, d=4096, E=8, top_k=2, G=4, d_ff=14336,
                           dtype="bf16", zipf_s=1.0, norm_topk=1),
    # fine-grained layer, 60 experts in 15 groups of 4 (the paper's E=60, 4-way case)
    "fine": LayerConfig("fine", T=8192, d=2048, E=60, top_k=4, G=15, d_ff=1408,
                        dtype="bf16", zipf_s=1.2),
    # heavy skew with two always-on shared experts
    "heavy": LayerConfig("heavy", T=16384, d=2048, E=64, top_k=6, G=16, d_ff=1408,
                         dtype="bf16", zipf_s=1.5, n_shared=2, d_ff_shared_each=1408),
    # decode-sized batch: a tiny, weight-streaming grouped GEMM
    "decode": LayerConfig("decode", T=64, d=2048, E=64, top_k=6, G=8, d_ff=1408,
                          dtype="bf16", zipf_s=1.2),
    # the fine-grained layer under partial brownout at the paper's threshold 0.4
    "partial": LayerConfig("partial", T=8192, d=2048, E=60, top_k=4, G=15, d_ff=1408,
                           dtype="bf16", zipf_s=1.2, theta=0.4),
}


def scaled(cfg: LayerConfig, **kw) -> LayerConfig:
    """A same-distribution copy of ``cfg`` at other sizes (for fast parity cases)."""
    return cfg.with_(name=cfg.name + "-" + "-".join(f"{k}{v}" for k, v in kw.items()), **kw)


# ---------------------------------------------------------------------------
# bf16 helpers (storage format only)

def _bf16_chunk(c: np.ndarray) -> np.ndarray:
    lsb = (c >> 16) & 1
    r = (c + np.uint32(0x7FFF) + lsb) >> 16
    nan = (c & 0x7FFFFFFF) > 0x7F800000
    if nan.any():
        r = np.where(nan, (c >> 16) | 0x40, r)
    return r.astype(np.uint16)


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 with round-to-nearest-even; returns uint16 bit patterns."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    flat_u = a.view(np.uint32).reshape(-1)
    out = np.empty(a.shape, dtype=np.uint16)
    flat_o = out.reshape(-1)
    step = 1 << 22
    starts = range(0, flat_u.size, step)

    def work(s):
        flat_o[s:s + step] = _bf16_chunk(flat_u[s:s + step])

    if flat_u.size <= step:
        for s in starts:
            work(s)
    else:
        import concurrent.futures as cf
        with cf.ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1)) as ex:
            list(ex.map(work, starts))
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to float32 (exact)."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def bf16_round_bits(a: np.ndarray) -> np.ndarray:
    return f32_to_bf16_bits(a)


# ---------------------------------------------------------------------------

@dataclasses.dataclass
class Layer:
    """One materialised workload.

    Float tensors are held in their storage format: float32 arrays for "f32"
    configurations, uint16 bf16 bit patterns for "bf16" ones. ``f32(name)``
    gives the exact float32 widening that the oracle consumes.
    """
    cfg: LayerConfig
    seed: int
    e2g: np.ndarray          # [E] int32, group of each expert
    bias: np.ndarray         # [E] float32, ln of the Zipf law
    x: np.ndarray            # [T, d]
    w_router: np.ndarray     # [E, d]
    w_gate: np.ndarray       # [G, d_ff, d]
    w_up: np.ndarray         # [G, d_ff, d]
    w_down: np.ndarray       # [G, d, d_ff]
    w_gate_sh: Optional[np.ndarray] = None   # [1, d_ff_shared, d]
    w_up_sh: Optional[np.ndarray] = None
    w_down_sh: Optional[np.ndarray] = None   # [1, d, d_ff_shared]

    def f32(self, name: str) -> np.ndarray:
        a = getattr(self, name)
        if a is None:
            return None
        if self.cfg.dtype == "f32":
            return a
        return bf16_bits_to_f32(a)


def _normal(rng: np.random.Generator, shape, std: float, dtype: str) -> np.ndarray:
    a = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        a *= np.float32(std)
    if dtype == "bf16":
        return f32_to_bf16_bits(a)
    return a


def balanced_map(perm: np.ndarray, E: int, G: int) -> np.ndarray:
    """Expert perm[i] -> group floor(i*G/E)."""
    e2g = np.empty(E, dtype=np.int32)
    for i in range(E):
        e2g[perm[i]] = (i * G) // E
    return e2g


def sequential_map(E: int, experts_per_group: int) -> np.ndarray:
    """Index-order grouping of the baseline system: experts 0..k-1 form group 0, etc."""
    return (np.arange(E, dtype=np.int32) // experts_per_group).astype(np.int32)


def zipf_bias(rank_perm: np.ndarray, s: float) -> np.ndarray:
    rho = 1.0 + rank_perm.astype(np.float64)
    q = rho ** (-s)
    q /= q.sum()
    return np.log(q).astype(np.float32)


def make_layer(cfg: LayerConfig, seed: int, *, with_weights: bool = True) -> Layer:
    """Draw one workload for ``cfg`` from ``seed`` (see module docstring)."""
    rng = np.random.default_rng(seed)
    E, G, d, T, f = cfg.E, cfg.G, cfg.d, cfg.T, cfg.d_ff
    map_perm = rng.permutation(E)
    rank_perm = rng.permutation(E)
    e2g = balanced_map(map_perm, E, G)
    bias = zipf_bias(rank_perm, cfg.zipf_s)
    x = _normal(rng, (T, d), 1.0, cfg.dtype)
    rstd = cfg.router_std if cfg.router_std is not None else 1.0 / math.sqrt(d)
    w_router = _normal(rng, (E, d), rstd, cfg.dtype)
    wstd = 1.0 / math.sqrt(d)
    if with_weights:
        w_gate = _normal(rng, (G, f, d), wstd, cfg.dtype)
        w_up = _normal(rng, (G, f, d), wstd, cfg.dtype)
        w_down = _normal(rng, (G, d, f), wstd, cfg.dtype)
    else:
        w_gate = w_up = w_down = None
    sh = (None, None, None)
    if cfg.n_shared and with_weights:
        fs = cfg.d_ff_shared
        sh = (_normal(rng, (1, fs, d), wstd, cfg.dtype),
              _normal(rng, (1, fs, d), wstd, cfg.dtype),
              _normal(rng, (1, d, fs), wstd, cfg.dtype))
    return Layer(cfg, seed, e2g, bias, x, w_router, w_gate, w_up, w_down, *sh)


def zipf_freq(L: Layer) -> np.ndarray:
    """The Zipf law behind the skew bias: the stand-in calibration frequencies."""
    q = np.exp(L.bias.astype(np.float64))
    return q / q.sum()


def expert_weights(L: Layer, e: int):
    """Original FFN of expert e: (w_gate [d_ff, d], w_up [d_ff, d], w_down [d, d_ff])."""
    cfg = L.cfg
    rng = np.random.default_rng([L.seed, 1_000_000 + int(e)])
    wstd = 1.0 / math.sqrt(cfg.d)
    return (_normal(rng, (cfg.d_ff, cfg.d), wstd, cfg.dtype),
            _normal(rng, (cfg.d_ff, cfg.d), wstd, cfg.dtype),
            _normal(rng, (cfg.d, cfg.d_ff), wstd, cfg.dtype))


def segment_layer(L: Layer, e2s: np.ndarray, segments) -> Layer:
    """The layer over a segment map: segment s is ("expert", e) with expert e's
    original FFN or ("united", g) with united expert g; e2s replaces the map."""
    parts = [expert_weights(L, i) if kind == "expert" else (L.w_gate[i], L.w_up[i], L.w_down[i])
             for kind, i in segments]
    wg, wu, wd = (np.stack([p[j] for p in parts]) for j in range(3))
    cfg = L.cfg.with_(G=len(segments))
    return dataclasses.replace(L, cfg=cfg, e2g=np.asarray(e2s, dtype=np.int32), w_gate=wg, w_up=wu, w_down=wd)


def tp_share(L: Layer, P: int, r: int) -> Layer:
    """Rank r's share of the layer under P-way tensor parallelism: hidden
    columns [r*d_ff/P, (r+1)*d_ff/P) of every united expert and of each shared
    expert. Same tokens, router, bias and map."""
    cfg = L.cfg
    if P < 1 or not 0 <= r < P or cfg.d_ff % P or (cfg.n_shared and cfg.d_ff_shared_each % P):
        raise ValueError(f"d_ff={cfg.d_ff} (shared {cfg.d_ff_shared_each}) does not split {P} ways")
    q = cfg.d_ff // P
    cols = slice(r * q, (r + 1) * q)
    kw = dict(w_gate=np.ascontiguousarray(L.w_gate[:, cols, :]),
              w_up=np.ascontiguousarray(L.w_up[:, cols, :]),
              w_down=np.ascontiguousarray(L.w_down[:, :, cols]))
    ncfg = cfg.with_(name=f"{cfg.name}-tp{P}r{r}", d_ff=q)
    if cfg.n_shared:
        n, qs = cfg.n_shared, cfg.d_ff_shared_each // P
        sc = slice(r * qs, (r + 1) * qs)
        d = cfg.d
        kw.update(w_gate_sh=np.ascontiguousarray(L.w_gate_sh.reshape(n, -1, d)[:, sc, :].reshape(1, n * qs, d)),
                  w_up_sh=np.ascontiguousarray(L.w_up_sh.reshape(n, -1, d)[:, sc, :].reshape(1, n * qs, d)),
                  w_down_sh=np.ascontiguousarray(L.w_down_sh.reshape(d, n, -1)[:, :, sc].reshape(1, d, n * qs)))
        ncfg = ncfg.with_(d_ff_shared_each=qs)
    return dataclasses.replace(L, cfg=ncfg, **kw)


def ep_groups(G: int, P: int, r: int):
    """Rank r's united experts [g0, g1) under P-way expert parallelism."""
    if P < 1 or not 0 <= r < P:
        raise ValueError("rank out of range")
    return (r * G) // P, ((r + 1) * G) // P
