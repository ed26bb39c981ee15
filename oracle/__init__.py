"""CPU oracle of the grouped (full-brownout) MoE layer forward.

TEST INFRASTRUCTURE ONLY: the test-suite, the smoke check and the benchmark's
CPU-baseline leg may use it; the product library never does. It shares no
code with the HIP path. The arithmetic lives in ``bmoe_oracle.c`` (double
precision, ascending-index sums, float at stage boundaries); this module only
builds that file with gcc and marshals numpy arrays into it.

Stages (same split as the layer's four calls):
  router_logits      gate logits in double                     (Sec. 2.1)
  route_from_logits  softmax, top-k, map substitution, merge   (Sec. 2.1, Eq. 2, Sec. 4.3-4.4)
  dispatch           group histogram, prefix, stable permutation
  ffn                grouped SwiGLU FFN over united experts
  combine            gate-weighted sum back in token order
  layer              all of the above, plus shared experts
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "bmoe_oracle.c")
_LIB = os.path.join(_HERE, "libbmoe_oracle.so")
MAX_E = 1024
MAX_K = 64


def build(force: bool = True, src: str = _SRC, out: str = _LIB) -> str:
    """Compile the oracle with gcc (-O2, OpenMP, strict IEEE: no fast-math, no FMA contraction)."""
    if force or not os.path.exists(out) or os.path.getmtime(out) < os.path.getmtime(src):
        tmp = out + ".tmp%d" % os.getpid()
        subprocess.run(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11",
                        "-fno-fast-math", "-ffp-contract=off", src, "-o", tmp, "-lm"],
                       check=True)
        os.replace(tmp, out)
    return out


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _f32(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float32)


def _i32(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.int32)


class Oracle:
    """ctypes view of one build of ``bmoe_oracle.c`` (the default build, or a test variant)."""

    def __init__(self, lib_path: str):
        lib = ctypes.CDLL(lib_path)
        P = ctypes.c_void_p
        I = ctypes.c_int
        lib.oracle_num_threads.restype = I
        lib.oracle_set_num_threads.argtypes = [I]
        lib.oracle_router_logits.argtypes = [P, P, P, I, I, I, P]
        lib.oracle_route_from_logits.argtypes = [P, P, I, I, I, I, P, P, P, P]
        lib.oracle_route_from_logits_f32.argtypes = [P, P, I, I, I, I, P, P, P, P]
        lib.oracle_dispatch.argtypes = [P, I, I, I, P, P, P, P]
        lib.oracle_dispatch.restype = I
        lib.oracle_gather_rows.argtypes = [P, P, I, I, P]
        lib.oracle_ffn.argtypes = [I, P, I, I, P, P, P, P, P, P]
        lib.oracle_combine.argtypes = [P, P, P, P, I, I, I, P]
        self.lib = lib
        self.path = lib_path

    def num_threads(self) -> int:
        return int(self.lib.oracle_num_threads())

    def set_num_threads(self, n: int) -> None:
        self.lib.oracle_set_num_threads(int(n))

    def router_logits(self, x, w_router, bias=None) -> np.ndarray:
        x, w, b = _f32(x), _f32(w_router), _f32(bias)
        T, d = x.shape
        E = w.shape[0]
        assert w.shape == (E, d)
        z = np.empty((T, E), dtype=np.float64)
        self.lib.oracle_router_logits(_p(x), _p(w), _p(b), T, d, E, _p(z))
        return z

    def route_from_logits(self, z, e2g, top_k: int, norm_topk: int = 0):
        """Selection on ``z`` (float64 logits, or float32 logits taken as exact values)."""
        e2g = _i32(e2g)
        T, E = z.shape
        assert E <= MAX_E and 1 <= top_k <= min(E, MAX_K)
        idx = np.empty((T, top_k), np.int32)
        w = np.empty((T, top_k), np.float32)
        sg = np.empty((T, top_k), np.int32)
        gate = np.empty((T, top_k), np.float32)
        if z.dtype == np.float32:
            z = np.ascontiguousarray(z)
            self.lib.oracle_route_from_logits_f32(_p(z), _p(e2g), T, E, top_k, int(norm_topk),
                                                  _p(idx), _p(w), _p(sg), _p(gate))
        else:
            z = np.ascontiguousarray(z, dtype=np.float64)
            self.lib.oracle_route_from_logits(_p(z), _p(e2g), T, E, top_k, int(norm_topk),
                                              _p(idx), _p(w), _p(sg), _p(gate))
        return dict(topk_idx=idx, topk_w=w, slot_group=sg, slot_gate=gate)

    def route(self, x, w_router, bias, e2g, top_k: int, norm_topk: int = 0):
        z = self.router_logits(x, w_router, bias)
        out = self.route_from_logits(z, e2g, top_k, norm_topk)
        out["logits"] = z
        return out

    def dispatch(self, slot_group, G: int):
        sg = _i32(slot_group)
        T, k = sg.shape
        counts = np.empty(G, np.int32)
        offsets = np.empty(G + 1, np.int32)
        perm = np.empty(max(T * k, 1), np.int32)
        slot_row = np.empty((T, k), np.int32)
        n = self.lib.oracle_dispatch(_p(sg), T, k, G, _p(counts), _p(offsets), _p(perm),
                                     _p(slot_row))
        return dict(counts=counts, offsets=offsets, perm_token=perm[:n].copy(),
                    slot_row=slot_row, N=int(n))

    def gather_rows(self, x, perm_token):
        x = _f32(x)
        perm = _i32(perm_token)
        N, d = perm.shape[0], x.shape[1]
        out = np.empty((N, d), np.float32)
        if N:
            self.lib.oracle_gather_rows(_p(x), _p(perm), N, d, _p(out))
        return out

    def ffn(self, offsets, a, w_gate, w_up, w_down, want_h: bool = False):
        offsets = _i32(offsets)
        a, wg, wu, wd = _f32(a), _f32(w_gate), _f32(w_up), _f32(w_down)
        n_seg, d_ff, d = wg.shape
        assert wu.shape == wg.shape and wd.shape == (n_seg, d, d_ff)
        assert offsets.shape == (n_seg + 1,)
        assert offsets[0] == 0, "segments start at row 0"
        N = int(offsets[-1])
        assert a.shape[1] == d and a.shape[0] >= N
        y = np.empty((N, d), np.float32)
        h = np.empty((N, d_ff), np.float32) if want_h else None
        self.lib.oracle_ffn(n_seg, _p(offsets), d, d_ff, _p(a), _p(wg), _p(wu), _p(wd), _p(h),
                            _p(y))
        return (y, h) if want_h else y

    def combine(self, slot_row, slot_gate, y, y_shared=None, d: Optional[int] = None):
        sr, sg = _i32(slot_row), _f32(slot_gate)
        y, ysh = _f32(y), _f32(y_shared)
        T, k = sr.shape
        if d is None:
            d = y.shape[1] if y.ndim == 2 and y.shape[0] else ysh.shape[1]
        out = np.empty((T, d), np.float32)
        self.lib.oracle_combine(_p(sr), _p(sg), _p(y), _p(ysh), T, k, d, _p(out))
        return out

    def layer(self, layer_inputs, logits_in=None, want_intermediates: bool = False):
        """Whole layer forward for a ``workload.Layer`` (or any object with the same fields)."""
        L = layer_inputs
        cfg = L.cfg
        x = L.f32("x")
        if logits_in is None:
            r = self.route(x, L.f32("w_router"), L.bias, L.e2g, cfg.top_k, cfg.norm_topk)
        else:
            r = self.route_from_logits(logits_in, L.e2g, cfg.top_k, cfg.norm_topk)
        dsp = self.dispatch(r["slot_group"], cfg.G)
        x_perm = self.gather_rows(x, dsp["perm_token"])
        y, h = self.ffn(dsp["offsets"], x_perm, L.f32("w_gate"), L.f32("w_up"), L.f32("w_down"),
                        want_h=True)
        y_sh = None
        if cfg.n_shared:
            y_sh = self.ffn(np.array([0, cfg.T], np.int32), x, L.f32("w_gate_sh"),
                            L.f32("w_up_sh"), L.f32("w_down_sh"))
        out = self.combine(dsp["slot_row"], r["slot_gate"], y, y_sh, d=cfg.d)
        if not want_intermediates:
            return out
        res = dict(out=out, y=y, h=h, x_perm=x_perm, y_shared=y_sh)
        res.update(r)
        res.update(dsp)
        return res


_default: Optional[Oracle] = None


def default() -> Oracle:
    global _default
    if _default is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build(force=True)
        _default = Oracle(_LIB)
    return _default


def _fwd(name):
    def f(*a, **kw):
        return getattr(default(), name)(*a, **kw)
    f.__name__ = name
    f.__doc__ = getattr(Oracle, name).__doc__
    return f


num_threads = _fwd("num_threads")
set_num_threads = _fwd("set_num_threads")
router_logits = _fwd("router_logits")
route_from_logits = _fwd("route_from_logits")
route = _fwd("route")
dispatch = _fwd("dispatch")
gather_rows = _fwd("gather_rows")
ffn = _fwd("ffn")
combine = _fwd("combine")
layer = _fwd("layer")
