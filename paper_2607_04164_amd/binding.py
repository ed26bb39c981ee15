"""Python binding of libbrownout_moe (argument marshalling only).

Every function here checks tensor placement/dtype/shape, passes raw device
pointers and the current HIP stream to the C ABI declared in
``include/brownout_moe.h``, and raises ``BmoeError`` on a non-OK status. All
arithmetic runs in the library's HIP kernels; torch provides device memory and
streams. There is no fallback: without the built library every call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional, Tuple

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libbrownout_moe.so")

BMOE_F32, BMOE_BF16 = 0, 1
STAGE_ROUTE, STAGE_DISPATCH, STAGE_FFN, STAGE_COMBINE, STAGE_DOWN_COMBINE = 0, 1, 2, 3, 4
ROUTE_RECHECK_GAP = 1.0 / 16384.0
MAX_EXPERTS, MAX_TOPK = 256, 16

STATUS = {0: "BMOE_OK", 1: "BMOE_ERR_NULL", 2: "BMOE_ERR_SHAPE", 3: "BMOE_ERR_ALIGN",
          4: "BMOE_ERR_MAP", 5: "BMOE_ERR_UNSUPPORTED", 6: "BMOE_ERR_WORKSPACE", 7: "BMOE_ERR_HIP"}

EXPORTED = ("bmoe_validate", "bmoe_validate_map", "bmoe_workspace_bytes", "bmoe_status_str",
            "bmoe_version", "brownout_moe_route", "brownout_moe_dispatch", "brownout_moe_ffn",
            "brownout_moe_ffn_gate_up", "brownout_moe_ffn_down", "brownout_moe_combine",
            "brownout_moe_ffn_gather", "brownout_moe_ffn_gate_up_gather", "brownout_moe_united_init",
            "brownout_moe_distill_mse", "brownout_moe_ffn_ex", "bmoe_partial_segment_map", "brownout_moe_dispatch_noalloc", "brownout_moe_ffn_down_combine")
STATUS_CODES = {v: k for k, v in STATUS.items()}
DISTILL_WS_BYTES = 32768
DISPATCH_SCRATCH_BYTES = 1048576  # the array behind brownout_moe_dispatch_noalloc


class BmoeError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {STATUS.get(status, status)} ({status_str(status)})")


class Desc(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int32), ("d", ctypes.c_int32), ("E", ctypes.c_int32),
                ("top_k", ctypes.c_int32), ("G", ctypes.c_int32), ("d_ff", ctypes.c_int32),
                ("d_ff_shared", ctypes.c_int32), ("norm_topk", ctypes.c_int32),
                ("dtype", ctypes.c_int32)]

    @property
    def torch_dtype(self):
        return torch.bfloat16 if self.dtype == BMOE_BF16 else torch.float32

    def replace(self, **kw) -> "Desc":
        vals = {f: getattr(self, f) for f, _ in self._fields_}
        vals.update(kw)
        return Desc(**vals)


def make_desc(T, d, E, top_k, G, d_ff, d_ff_shared=0, norm_topk=0, dtype="bf16") -> Desc:
    dt = {"bf16": BMOE_BF16, "f32": BMOE_F32, BMOE_BF16: BMOE_BF16, BMOE_F32: BMOE_F32}[dtype]
    return Desc(int(T), int(d), int(E), int(top_k), int(G), int(d_ff), int(d_ff_shared),
                int(norm_topk), dt)


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load the HIP library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it first (python -c 'import __graft_entry__ as g; g.build()')")
    lib = ctypes.CDLL(path)
    P, I32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    DP = ctypes.POINTER(Desc)
    lib.bmoe_validate.argtypes = [DP]
    lib.bmoe_validate.restype = I32
    lib.bmoe_validate_map.argtypes = [P, I32, I32]
    lib.bmoe_validate_map.restype = I32
    lib.bmoe_workspace_bytes.argtypes = [DP, I32]
    lib.bmoe_workspace_bytes.restype = SZ
    lib.bmoe_status_str.argtypes = [I32]
    lib.bmoe_status_str.restype = ctypes.c_char_p
    lib.bmoe_version.restype = I32
    lib.brownout_moe_route.argtypes = [DP] + [P] * 11
    lib.brownout_moe_route.restype = I32
    lib.brownout_moe_dispatch.argtypes = [DP] + [P] * 8 + [SZ, P]
    lib.brownout_moe_dispatch.restype = I32
    lib.brownout_moe_dispatch_noalloc.argtypes = [DP] + [P] * 8
    lib.brownout_moe_dispatch_noalloc.restype = I32
    lib.brownout_moe_ffn.argtypes = [I32] * 5 + [P] * 8 + [SZ, P]
    lib.brownout_moe_ffn.restype = I32
    lib.brownout_moe_ffn_ex.argtypes = [I32] * 5 + [P] * 8 + [SZ, I32, P]
    lib.brownout_moe_ffn_ex.restype = I32
    lib.brownout_moe_ffn_gate_up.argtypes = [I32] * 5 + [P] * 6 + [SZ, P]
    lib.brownout_moe_ffn_gate_up.restype = I32
    lib.brownout_moe_ffn_down.argtypes = [I32] * 5 + [P] * 5 + [SZ, P]
    lib.brownout_moe_ffn_gather.argtypes = [I32] * 5 + [P, P, I32] + [P] * 7 + [SZ, P]
    lib.brownout_moe_ffn_gather.restype = I32
    lib.brownout_moe_ffn_gate_up_gather.argtypes = [I32] * 5 + [P, P, I32] + [P] * 5 + [SZ, P]
    lib.brownout_moe_ffn_gate_up_gather.restype = I32
    lib.brownout_moe_united_init.argtypes = [I32] * 5 + [P] * 8
    lib.brownout_moe_united_init.restype = I32
    lib.brownout_moe_distill_mse.argtypes = [I32] * 5 + [P] * 7 + [SZ, P]
    lib.brownout_moe_distill_mse.restype = I32
    lib.brownout_moe_ffn_down.restype = I32
    lib.brownout_moe_combine.argtypes = [DP] + [P] * 6
    lib.brownout_moe_combine.restype = I32
    lib.brownout_moe_ffn_down_combine.argtypes = [DP] + [P] * 10 + [SZ, P]
    lib.brownout_moe_ffn_down_combine.restype = I32
    lib.bmoe_partial_segment_map.argtypes = [P, P, I32, I32, ctypes.c_double, P, P, P, P]
    lib.bmoe_partial_segment_map.restype = I32
    _lib = lib
    return lib


def status_str(status: int) -> str:
    return load_library().bmoe_status_str(int(status)).decode()


def _check(status: int, where: str):
    if status != 0:
        raise BmoeError(status, where)


def validate(desc: Desc) -> int:
    return int(load_library().bmoe_validate(ctypes.byref(desc)))


def validate_map(e2g_host, E: int, G: int) -> int:
    import numpy as np
    a = np.ascontiguousarray(e2g_host, dtype=np.int32)
    return int(load_library().bmoe_validate_map(a.ctypes.data_as(ctypes.c_void_p), int(E), int(G)))


def workspace_bytes(desc: Desc, stage: int) -> int:
    return int(load_library().bmoe_workspace_bytes(ctypes.byref(desc), int(stage)))


def _p(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None) -> ctypes.c_void_p:
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _dev(t: torch.Tensor, name: str, dtype=None, shape=None):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    return t


def _empty(shape, dtype, device):
    return torch.empty(shape, dtype=dtype, device=device)


# ---------------------------------------------------------------------------
# the four calls

def route(desc: Desc, x: Optional[torch.Tensor], w_router: Optional[torch.Tensor],
          bias: Optional[torch.Tensor], e2g: torch.Tensor, *, logits_in: Optional[torch.Tensor] = None,
          want_logits: bool = False, out: Optional[Dict[str, torch.Tensor]] = None,
          stream=None) -> Dict[str, torch.Tensor]:
    T, E, k = desc.T, desc.E, desc.top_k
    dev = e2g.device
    _dev(e2g, "e2g", torch.int32, (E,))
    if logits_in is None:
        _dev(x, "x", desc.torch_dtype, (T, desc.d))
        _dev(w_router, "w_router", desc.torch_dtype, (E, desc.d))
        if bias is not None:
            _dev(bias, "bias", torch.float32, (E,))
    else:
        _dev(logits_in, "logits_in", torch.float32, (T, E))
    o = dict(out) if out else {}
    o.setdefault("topk_idx", _empty((T, k), torch.int32, dev))
    o.setdefault("topk_w", _empty((T, k), torch.float32, dev))
    o.setdefault("slot_group", _empty((T, k), torch.int32, dev))
    o.setdefault("slot_gate", _empty((T, k), torch.float32, dev))
    if want_logits:
        o.setdefault("logits", _empty((T, E), torch.float32, dev))
    st = load_library().brownout_moe_route(
        ctypes.byref(desc), _p(x), _p(w_router), _p(bias), _p(logits_in), _p(e2g), _p(o["topk_idx"]),
        _p(o["topk_w"]), _p(o["slot_group"]), _p(o["slot_gate"]), _p(o.get("logits")), _stream(stream))
    _check(st, "brownout_moe_route")
    return o


def dispatch(desc: Desc, slot_group: torch.Tensor, x: Optional[torch.Tensor], workspace: torch.Tensor, *,
             out: Optional[Dict[str, torch.Tensor]] = None, copy_rows: bool = True,
             stream=None) -> Dict[str, torch.Tensor]:
    """copy_rows=False: the permutation only (no x_perm; x may be None), for
    the FFN that gathers its rows itself (ffn_gather)."""
    T, k, G, d = desc.T, desc.top_k, desc.G, desc.d
    dev = slot_group.device
    _dev(slot_group, "slot_group", torch.int32, (T, k))
    if copy_rows or x is not None:
        _dev(x, "x", desc.torch_dtype, (T, d))
    _dev(workspace, "workspace")
    o = dict(out) if out else {}
    o.setdefault("counts", _empty((G,), torch.int32, dev))
    o.setdefault("offsets", _empty((G + 1,), torch.int32, dev))
    o.setdefault("perm_token", _empty((max(T * k, 1),), torch.int32, dev))
    o.setdefault("slot_row", _empty((T, k), torch.int32, dev))
    if copy_rows:
        o.setdefault("x_perm", _empty((max(T * k, 1), d), desc.torch_dtype, dev))
    st = load_library().brownout_moe_dispatch(
        ctypes.byref(desc), _p(slot_group), _p(x), _p(o["counts"]), _p(o["offsets"]),
        _p(o["perm_token"]), _p(o["slot_row"]), _p(o["x_perm"]) if copy_rows else None, _p(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream))
    _check(st, "brownout_moe_dispatch")
    return o


def dispatch_noalloc(desc: Desc, slot_group: torch.Tensor, x: Optional[torch.Tensor], *,
                     out: Optional[Dict[str, torch.Tensor]] = None, copy_rows: bool = True,
                     stream=None) -> Dict[str, torch.Tensor]:
    """dispatch on the library's own per-device workspace array (the call
    allocates nothing on the device; pass every output in ``out`` to keep this
    wrapper from allocating them)."""
    T, k, G, d = desc.T, desc.top_k, desc.G, desc.d
    dev = slot_group.device
    _dev(slot_group, "slot_group", torch.int32, (T, k))
    if copy_rows or x is not None:
        _dev(x, "x", desc.torch_dtype, (T, d))
    o = dict(out) if out else {}
    o.setdefault("counts", _empty((G,), torch.int32, dev))
    o.setdefault("offsets", _empty((G + 1,), torch.int32, dev))
    o.setdefault("perm_token", _empty((max(T * k, 1),), torch.int32, dev))
    o.setdefault("slot_row", _empty((T, k), torch.int32, dev))
    if copy_rows:
        o.setdefault("x_perm", _empty((max(T * k, 1), d), desc.torch_dtype, dev))
    st = load_library().brownout_moe_dispatch_noalloc(
        ctypes.byref(desc), _p(slot_group), _p(x), _p(o["counts"]), _p(o["offsets"]),
        _p(o["perm_token"]), _p(o["slot_row"]), _p(o["x_perm"]) if copy_rows else None, _stream(stream))
    _check(st, "brownout_moe_dispatch_noalloc")
    return o


def new_dispatch_workspace(desc: Desc, device) -> torch.Tensor:
    """An all-zero workspace of the size dispatch needs (kept zero by every call)."""
    n = workspace_bytes(desc, STAGE_DISPATCH)
    return torch.zeros((n + 255) // 256 * 256, dtype=torch.uint8, device=device)


def new_ffn_workspace(desc: Desc, device) -> Optional[torch.Tensor]:
    """The FFN stream-K workspace for this device (None when the layer has no
    use for one: fp32, or no device)."""
    n = workspace_bytes(desc, STAGE_FFN)
    return torch.empty((n + 255) // 256 * 256, dtype=torch.uint8, device=device) if n else None


def _ws(ws: Optional[torch.Tensor]):
    if ws is None:
        return None, 0
    _dev(ws, "workspace", torch.uint8)
    return _p(ws), ws.numel()


def _ffn_checks(offsets, a_rows, dt, n_seg, d, d_ff):
    dtype = {torch.bfloat16: BMOE_BF16, torch.float32: BMOE_F32}.get(dt)
    if dtype is None:
        raise ValueError(f"unsupported dtype {dt}")
    _dev(offsets, "offsets", torch.int32, (n_seg + 1,))
    return dtype


def ffn(offsets: torch.Tensor, a: torch.Tensor, w_gate: torch.Tensor, w_up: torch.Tensor,
        w_down: torch.Tensor, *, h: Optional[torch.Tensor] = None, y: Optional[torch.Tensor] = None,
        workspace: Optional[torch.Tensor] = None, split_min_idle: Optional[int] = None, stream=None):
    """Both grouped GEMMs: returns (y, h). workspace: optional uint8 device
    tensor of at least workspace_bytes(desc, STAGE_FFN) bytes (stream-K);
    split_min_idle: the stream-K split threshold (None: the library default)."""
    n_seg, d_ff, d = w_gate.shape
    rows_cap, dt = a.shape[0], a.dtype
    dtype = _ffn_checks(offsets, rows_cap, dt, n_seg, d, d_ff)
    _dev(a, "a", dt, (rows_cap, d))
    _dev(w_gate, "w_gate", dt, (n_seg, d_ff, d))
    _dev(w_up, "w_up", dt, (n_seg, d_ff, d))
    _dev(w_down, "w_down", dt, (n_seg, d, d_ff))
    h = _dev(h, "h", dt, (rows_cap, d_ff)) if h is not None else _empty((rows_cap, d_ff), dt, a.device)
    y = _dev(y, "y", dt, (rows_cap, d)) if y is not None else _empty((rows_cap, d), dt, a.device)
    wsp, wsn = _ws(workspace)
    if split_min_idle is None:
        st = load_library().brownout_moe_ffn(dtype, n_seg, rows_cap, d, d_ff, _p(offsets), _p(a), _p(w_gate),
                                             _p(w_up), _p(w_down), _p(h), _p(y), wsp, wsn, _stream(stream))
        _check(st, "brownout_moe_ffn")
    else:
        st = load_library().brownout_moe_ffn_ex(dtype, n_seg, rows_cap, d, d_ff, _p(offsets), _p(a), _p(w_gate),
                                                _p(w_up), _p(w_down), _p(h), _p(y), wsp, wsn, int(split_min_idle),
                                                _stream(stream))
        _check(st, "brownout_moe_ffn_ex")
    return y, h


def ffn_gate_up(offsets, a, w_gate, w_up, *, h=None, workspace=None, stream=None):
    n_seg, d_ff, d = w_gate.shape
    rows_cap, dt = a.shape[0], a.dtype
    dtype = _ffn_checks(offsets, rows_cap, dt, n_seg, d, d_ff)
    _dev(a, "a", dt, (rows_cap, d))
    _dev(w_gate, "w_gate", dt, (n_seg, d_ff, d))
    _dev(w_up, "w_up", dt, (n_seg, d_ff, d))
    h = _dev(h, "h", dt, (rows_cap, d_ff)) if h is not None else _empty((rows_cap, d_ff), dt, a.device)
    wsp, wsn = _ws(workspace)
    st = load_library().brownout_moe_ffn_gate_up(dtype, n_seg, rows_cap, d, d_ff, _p(offsets), _p(a),
                                                 _p(w_gate), _p(w_up), _p(h), wsp, wsn, _stream(stream))
    _check(st, "brownout_moe_ffn_gate_up")
    return h


def ffn_gather(offsets: torch.Tensor, a_rows: torch.Tensor, a: torch.Tensor, w_gate: torch.Tensor,
               w_up: torch.Tensor, w_down: torch.Tensor, *, h=None, y=None, workspace=None, stream=None):
    """ffn with the gate/up activations gathered: row r reads a[a_rows[r]]
    (a_rows: the dispatch's perm_token, a: x). rows_cap = a_rows.numel().
    Returns (y, h)."""
    n_seg, d_ff, d = w_gate.shape
    rows_cap, dt = a_rows.numel(), a.dtype
    dtype = _ffn_checks(offsets, rows_cap, dt, n_seg, d, d_ff)
    _dev(a_rows, "a_rows", torch.int32, (rows_cap,))
    _dev(a, "a", dt)
    if a.dim() != 2 or a.shape[1] != d:
        raise ValueError(f"a must be [rows, {d}]")
    _dev(w_gate, "w_gate", dt, (n_seg, d_ff, d))
    _dev(w_up, "w_up", dt, (n_seg, d_ff, d))
    _dev(w_down, "w_down", dt, (n_seg, d, d_ff))
    h = _dev(h, "h", dt, (rows_cap, d_ff)) if h is not None else _empty((rows_cap, d_ff), dt, a.device)
    y = _dev(y, "y", dt, (rows_cap, d)) if y is not None else _empty((rows_cap, d), dt, a.device)
    wsp, wsn = _ws(workspace)
    st = load_library().brownout_moe_ffn_gather(dtype, n_seg, rows_cap, d, d_ff, _p(offsets), _p(a_rows),
                                                a.shape[0], _p(a), _p(w_gate), _p(w_up), _p(w_down), _p(h),
                                                _p(y), wsp, wsn, _stream(stream))
    _check(st, "brownout_moe_ffn_gather")
    return y, h


def ffn_gate_up_gather(offsets, a_rows, a, w_gate, w_up, *, h=None, workspace=None, stream=None):
    n_seg, d_ff, d = w_gate.shape
    rows_cap, dt = a_rows.numel(), a.dtype
    dtype = _ffn_checks(offsets, rows_cap, dt, n_seg, d, d_ff)
    _dev(a_rows, "a_rows", torch.int32, (rows_cap,))
    _dev(a, "a", dt)
    if a.dim() != 2 or a.shape[1] != d:
        raise ValueError(f"a must be [rows, {d}]")
    _dev(w_gate, "w_gate", dt, (n_seg, d_ff, d))
    _dev(w_up, "w_up", dt, (n_seg, d_ff, d))
    h = _dev(h, "h", dt, (rows_cap, d_ff)) if h is not None else _empty((rows_cap, d_ff), dt, a.device)
    wsp, wsn = _ws(workspace)
    st = load_library().brownout_moe_ffn_gate_up_gather(dtype, n_seg, rows_cap, d, d_ff, _p(offsets), _p(a_rows),
                                                        a.shape[0], _p(a), _p(w_gate), _p(w_up), _p(h), wsp, wsn,
                                                        _stream(stream))
    _check(st, "brownout_moe_ffn_gate_up_gather")
    return h


# ---------------------------------------------------------------------------
# grouping search: expert outputs on calibration tokens, united init, errors

def all_tokens_rows(n: int, T: int, device) -> Tuple[torch.Tensor, torch.Tensor]:
    """(offsets, a_rows) that run n FFNs over the same T tokens with
    ffn_gather: segment s covers rows s*T .. s*T+T-1, row r reads token r mod T."""
    offsets = torch.arange(n + 1, dtype=torch.int32, device=device) * T
    a_rows = torch.arange(T, dtype=torch.int32, device=device).repeat(n)
    return offsets, a_rows


def ffn_all_tokens(x: torch.Tensor, w_gate, w_up, w_down, *, workspace=None, stream=None) -> torch.Tensor:
    """Every FFN of the stack on every token: [n*T, d], rows s*T + t = FFN_s(x_t)."""
    n, T = w_gate.shape[0], x.shape[0]
    offsets, a_rows = all_tokens_rows(n, T, x.device)
    y, _ = ffn_gather(offsets, a_rows, x, w_gate, w_up, w_down, workspace=workspace, stream=stream)
    return y


def united_init(e2g: torch.Tensor, G: int, w_gate_e, w_up_e, w_down_e, *, out=None, stream=None):
    """Parameter-average starting weights of the G united experts: (w_gate, w_up, w_down)."""
    E, f, d = w_gate_e.shape
    dt = w_gate_e.dtype
    dtype = {torch.bfloat16: BMOE_BF16, torch.float32: BMOE_F32}[dt]
    _dev(e2g, "e2g", torch.int32, (E,))
    _dev(w_gate_e, "w_gate_e", dt, (E, f, d))
    _dev(w_up_e, "w_up_e", dt, (E, f, d))
    _dev(w_down_e, "w_down_e", dt, (E, d, f))
    if out is None:
        out = (_empty((G, f, d), dt, e2g.device), _empty((G, f, d), dt, e2g.device), _empty((G, d, f), dt, e2g.device))
    for t, shp, nm in zip(out, ((G, f, d), (G, f, d), (G, d, f)), ("w_gate_u", "w_up_u", "w_down_u")):
        _dev(t, nm, dt, shp)
    st = load_library().brownout_moe_united_init(dtype, E, G, d, f, _p(e2g), _p(w_gate_e), _p(w_up_e), _p(w_down_e),
                                                 _p(out[0]), _p(out[1]), _p(out[2]), _stream(stream))
    _check(st, "brownout_moe_united_init")
    return out


def distill_mse(e2g: torch.Tensor, w_freq: torch.Tensor, y_expert: torch.Tensor, y_united: torch.Tensor, T: int,
                *, workspace: Optional[torch.Tensor] = None, out=None, stream=None):
    """(mse [G] float64, total [] float64) of Eq. 5-6 from the experts' outputs
    [E*T, d] and the united experts' outputs [G*T, d] on T tokens."""
    E = e2g.numel()
    G = y_united.shape[0] // T if T else 0
    d = y_expert.shape[1]
    dt = y_expert.dtype
    dtype = {torch.bfloat16: BMOE_BF16, torch.float32: BMOE_F32}[dt]
    _dev(e2g, "e2g", torch.int32, (E,))
    _dev(w_freq, "w_freq", torch.float32, (E,))
    _dev(y_expert, "y_expert", dt, (E * T, d))
    _dev(y_united, "y_united", dt, (G * T, d))
    if workspace is None:
        workspace = torch.empty(DISTILL_WS_BYTES, dtype=torch.uint8, device=e2g.device)
    _dev(workspace, "workspace", torch.uint8)
    mse, total = out if out is not None else (torch.zeros(G, dtype=torch.float64, device=e2g.device),
                                              torch.zeros((), dtype=torch.float64, device=e2g.device))
    st = load_library().brownout_moe_distill_mse(dtype, E, G, T, d, _p(e2g), _p(w_freq), _p(y_expert),
                                                 _p(y_united), _p(mse), _p(total), _p(workspace),
                                                 workspace.numel(), _stream(stream))
    _check(st, "brownout_moe_distill_mse")
    return mse, total


def ffn_down(offsets, h, w_down, *, y=None, workspace=None, stream=None):
    n_seg, d, d_ff = w_down.shape
    rows_cap, dt = h.shape[0], h.dtype
    dtype = _ffn_checks(offsets, rows_cap, dt, n_seg, d, d_ff)
    _dev(h, "h", dt, (rows_cap, d_ff))
    _dev(w_down, "w_down", dt, (n_seg, d, d_ff))
    y = _dev(y, "y", dt, (rows_cap, d)) if y is not None else _empty((rows_cap, d), dt, h.device)
    wsp, wsn = _ws(workspace)
    st = load_library().brownout_moe_ffn_down(dtype, n_seg, rows_cap, d, d_ff, _p(offsets), _p(h),
                                              _p(w_down), _p(y), wsp, wsn, _stream(stream))
    _check(st, "brownout_moe_ffn_down")
    return y


def combine(desc: Desc, slot_row: torch.Tensor, slot_gate: torch.Tensor, y_perm: torch.Tensor,
            y_shared: Optional[torch.Tensor] = None, *, out: Optional[torch.Tensor] = None, stream=None):
    T, k, d = desc.T, desc.top_k, desc.d
    _dev(slot_row, "slot_row", torch.int32, (T, k))
    _dev(slot_gate, "slot_gate", torch.float32, (T, k))
    _dev(y_perm, "y_perm", desc.torch_dtype)
    if y_perm.shape[0] < T * k or y_perm.shape[1] != d:
        raise ValueError("y_perm must be [>= T*k, d]")
    if y_shared is not None:
        _dev(y_shared, "y_shared", desc.torch_dtype, (T, d))
    out = _dev(out, "out", desc.torch_dtype, (T, d)) if out is not None else _empty((T, d), desc.torch_dtype, slot_row.device)
    st = load_library().brownout_moe_combine(ctypes.byref(desc), _p(slot_row), _p(slot_gate), _p(y_perm),
                                             _p(y_shared), _p(out), _stream(stream))
    _check(st, "brownout_moe_combine")
    return out


def new_down_combine_workspace(desc: Desc, device) -> torch.Tensor:
    """The all-zero counter workspace of ffn_down_combine (kept zero by every call)."""
    n = workspace_bytes(desc, STAGE_DOWN_COMBINE)
    return torch.zeros((n + 255) // 256 * 256, dtype=torch.uint8, device=device)


def ffn_down_combine(desc: Desc, offsets, h, w_down, perm_token, slot_row, slot_gate, workspace,
                     y_shared=None, *, y=None, out=None, stream=None):
    """The down projection with the combine folded into its epilogue:
    returns (y, out), bit-identical to ffn_down (without a stream-K workspace)
    followed by combine."""
    T, k, d, G, f = desc.T, desc.top_k, desc.d, desc.G, desc.d_ff
    dt = desc.torch_dtype
    rows = max(T * k, 1)
    _dev(offsets, "offsets", torch.int32, (G + 1,))
    _dev(h, "h", dt, (rows, f))
    _dev(w_down, "w_down", dt, (G, d, f))
    _dev(perm_token, "perm_token", torch.int32, (rows,))
    _dev(slot_row, "slot_row", torch.int32, (T, k))
    _dev(slot_gate, "slot_gate", torch.float32, (T, k))
    _dev(workspace, "workspace", torch.uint8)
    if y_shared is not None:
        _dev(y_shared, "y_shared", dt, (T, d))
    y = _dev(y, "y", dt, (rows, d)) if y is not None else _empty((rows, d), dt, h.device)
    out = _dev(out, "out", dt, (T, d)) if out is not None else _empty((T, d), dt, h.device)
    st = load_library().brownout_moe_ffn_down_combine(
        ctypes.byref(desc), _p(offsets), _p(h), _p(w_down), _p(y), _p(perm_token), _p(slot_row), _p(slot_gate),
        _p(y_shared), _p(out), _p(workspace), workspace.numel(), _stream(stream))
    _check(st, "brownout_moe_ffn_down_combine")
    return y, out


# ---------------------------------------------------------------------------

# top_k from which LayerForward takes the fused gather by default
FUSED_GATHER_MIN_TOP_K = 3


class LayerForward:
    """One grouped MoE layer with its weights and every intermediate buffer
    allocated once, so a forward enqueues only the library's kernels.

    weights: dict with w_router [E,d], bias [E] (float or None), e2g [E] int32,
    w_gate/w_up [G,d_ff,d], w_down [G,d,d_ff], and optionally w_gate_sh/w_up_sh
    [1,d_ff_shared,d], w_down_sh [1,d,d_ff_shared] (all device tensors).

    Weights, buffers and workspaces are checked once here and their pointers
    marshalled once; a call checks only x and looks up the current stream, so
    the host cost per call stays a few microseconds (decode-sized layers take
    less GPU time than the checks of the free functions).

    fused_gather=True: dispatch writes only the permutation and the gate/up
    GEMM gathers its rows from x (no x_perm buffer); ffn and ffn_gate_up then
    take x. Results are bit-identical to the unfused path. None (the default)
    takes it when top_k >= FUSED_GATHER_MIN_TOP_K (and x is below 4 GiB, the
    gather's addressing limit): x_perm then holds top_k
    copies of x's rows, and writing and re-reading it costs more than the
    GEMM's row gather (fine, heavy, decode and partial-brownout workloads,
    top-4 and top-6: layer 2-4 % faster); at top-2 the two paths time alike
    and the four calls are kept.

    fold_combine=True: the combine runs in the down projection's epilogue
    (brownout_moe_ffn_down_combine; its tiles are never split, so the layer
    equals the unfused layer without the stream-K workspace, bit for bit).

    concurrent_shared=True (layers with shared experts): a forward starts the
    shared-expert FFN on a side stream of the layer's own (default priority)
    as soon as x is ready and joins it before the combine; the routed path
    runs meanwhile on the caller's stream. The shared FFN then runs without
    the stream-K workspace (whole tiles; with a split its last bits could
    differ from the one-stream forward, which splits where the workspace
    allows).
    """

    def __init__(self, desc: Desc, weights: Dict[str, torch.Tensor], device="cuda", stream_k: bool = True,
                 fused_gather: Optional[bool] = None, fold_combine: bool = False, concurrent_shared: bool = True):
        self.desc = desc
        self.w = weights
        if fused_gather is None:
            # (the gathered copies address x with 32-bit byte offsets)
            x_bytes = desc.T * desc.d * (2 if desc.dtype == BMOE_BF16 else 4)
            fused_gather = desc.top_k >= FUSED_GATHER_MIN_TOP_K and x_bytes < (1 << 32)
        self.fused_gather = bool(fused_gather)
        self.fold_combine = fold_combine
        _check(validate(desc), "bmoe_validate")
        T, k, d, G, E = desc.T, desc.top_k, desc.d, desc.G, desc.E
        dt = desc.torch_dtype
        rows = max(T * k, 1)
        self.bufs = {
            "route": {n: _empty((T, k), t, device) for n, t in
                      (("topk_idx", torch.int32), ("topk_w", torch.float32),
                       ("slot_group", torch.int32), ("slot_gate", torch.float32))},
            "dispatch": {"counts": _empty((G,), torch.int32, device),
                         "offsets": _empty((G + 1,), torch.int32, device),
                         "perm_token": _empty((rows,), torch.int32, device),
                         "slot_row": _empty((T, k), torch.int32, device)},
            "h": _empty((rows, desc.d_ff), dt, device),
            "y": _empty((rows, d), dt, device),
            "out": _empty((T, d), dt, device),
        }
        if not fused_gather:
            self.bufs["dispatch"]["x_perm"] = _empty((rows, d), dt, device)
        self.ws = new_dispatch_workspace(desc, device)
        self.ffn_ws = new_ffn_workspace(desc, device) if stream_k else None
        self.fold_ws = new_down_combine_workspace(desc, device) if fold_combine else None
        self._side = None
        if desc.d_ff_shared:
            self.bufs["h_sh"] = _empty((max(T, 1), desc.d_ff_shared), dt, device)
            self.bufs["y_sh"] = _empty((max(T, 1), d), dt, device)
            self.sh_offsets = torch.tensor([0, T], dtype=torch.int32, device=device)
            if concurrent_shared:
                # default priority, as every stream of the layer
                self._side = torch.cuda.Stream(device=device)
        self._plan()

    def _plan(self):
        """Checks every fixed tensor and marshals the fixed arguments of each call."""
        desc, w, b = self.desc, self.w, self.bufs
        T, k, d, G, E, f = desc.T, desc.top_k, desc.d, desc.G, desc.E, desc.d_ff
        dt = desc.torch_dtype
        dtype = BMOE_BF16 if dt == torch.bfloat16 else BMOE_F32
        _dev(w["w_router"], "w_router", dt, (E, d))
        _dev(w["e2g"], "e2g", torch.int32, (E,))
        if w.get("bias") is not None:
            _dev(w["bias"], "bias", torch.float32, (E,))
        _dev(w["w_gate"], "w_gate", dt, (G, f, d))
        _dev(w["w_up"], "w_up", dt, (G, f, d))
        _dev(w["w_down"], "w_down", dt, (G, d, f))
        ptr = lambda t: None if t is None else t.data_ptr()
        wsp, wsn = (ptr(self.ffn_ws), self.ffn_ws.numel()) if self.ffn_ws is not None else (None, 0)
        self._lib = load_library()
        self._desc_ref = ctypes.byref(desc)
        self._xshape, self._dt = (T, d), dt
        r, dp = b["route"], b["dispatch"]
        self._route_args = (ptr(w["w_router"]), ptr(w.get("bias")), None, ptr(w["e2g"]), ptr(r["topk_idx"]),
                            ptr(r["topk_w"]), ptr(r["slot_group"]), ptr(r["slot_gate"]), None)
        fused = self.fused_gather
        self._dispatch_args = (ptr(dp["counts"]), ptr(dp["offsets"]), ptr(dp["perm_token"]), ptr(dp["slot_row"]),
                               None if fused else ptr(dp["x_perm"]), ptr(self.ws), self.ws.numel())
        rows = max(T * k, 1)
        # fused: (.., offsets, a_rows, a_count) then x's pointer at call time
        a_src = (ptr(dp["perm_token"]), T) if fused else (ptr(dp["x_perm"]),)
        self._gate_up_args = (dtype, G, rows, d, f, ptr(dp["offsets"]), *a_src, ptr(w["w_gate"]),
                              ptr(w["w_up"]), ptr(b["h"]), wsp, wsn)
        self._down_args = (dtype, G, rows, d, f, ptr(dp["offsets"]), ptr(b["h"]), ptr(w["w_down"]), ptr(b["y"]),
                           wsp, wsn)
        self._ffn_args = (dtype, G, rows, d, f, ptr(dp["offsets"]), *a_src, ptr(w["w_gate"]),
                          ptr(w["w_up"]), ptr(w["w_down"]), ptr(b["h"]), ptr(b["y"]), wsp, wsn)
        self._a_at = 8 if fused else None  # where x's pointer goes in the fused argument lists
        self._combine_args = (ptr(dp["slot_row"]), ptr(r["slot_gate"]), ptr(b["y"]),
                              ptr(b["y_sh"]) if desc.d_ff_shared else None, ptr(b["out"]))
        if self.fold_combine:
            self._down_combine_args = (ptr(dp["offsets"]), ptr(b["h"]), ptr(w["w_down"]), ptr(b["y"]),
                                       ptr(dp["perm_token"]), ptr(dp["slot_row"]), ptr(r["slot_gate"]),
                                       ptr(b["y_sh"]) if desc.d_ff_shared else None, ptr(b["out"]),
                                       ptr(self.fold_ws), self.fold_ws.numel())
        if desc.d_ff_shared:
            fs = desc.d_ff_shared
            _dev(w["w_gate_sh"], "w_gate_sh", dt, (1, fs, d))
            _dev(w["w_up_sh"], "w_up_sh", dt, (1, fs, d))
            _dev(w["w_down_sh"], "w_down_sh", dt, (1, d, fs))
            self._shared_args = (dtype, 1, T, d, fs, ptr(self.sh_offsets), ptr(w["w_gate_sh"]),
                                 ptr(w["w_up_sh"]), ptr(w["w_down_sh"]), ptr(b["h_sh"]), ptr(b["y_sh"]), wsp, wsn)
            # on the side stream without the stream-K workspace, which the
            # routed FFN may be using at the same time (its tiles stay whole)
            self._shared_side_args = self._shared_args[:-2] + (None, 0)

    def _x(self, x) -> int:
        if not (isinstance(x, torch.Tensor) and x.is_cuda and x.dtype == self._dt
                and tuple(x.shape) == self._xshape and x.is_contiguous()):
            _dev(x, "x", self._dt, self._xshape)
        return x.data_ptr()

    @staticmethod
    def _s(stream) -> int:
        return (stream if stream is not None else torch.cuda.current_stream()).cuda_stream

    def route(self, x, stream=None):
        _check(self._lib.brownout_moe_route(self._desc_ref, self._x(x), *self._route_args[:2], None,
                                            *self._route_args[3:], self._s(stream)), "brownout_moe_route")
        return self.bufs["route"]

    def dispatch(self, x, stream=None):
        _check(self._lib.brownout_moe_dispatch(self._desc_ref, self.bufs["route"]["slot_group"].data_ptr(),
                                               self._x(x), *self._dispatch_args, self._s(stream)),
               "brownout_moe_dispatch")
        return self.bufs["dispatch"]

    def _fused_args(self, args, x):
        if x is None:
            raise ValueError("the fused-gather layer's FFN reads x: pass x")
        i = self._a_at
        return (*args[:i], self._x(x), *args[i:])

    def ffn(self, stream=None, x=None):
        if self.fused_gather:
            _check(self._lib.brownout_moe_ffn_gather(*self._fused_args(self._ffn_args, x), self._s(stream)),
                   "brownout_moe_ffn_gather")
        else:
            _check(self._lib.brownout_moe_ffn(*self._ffn_args, self._s(stream)), "brownout_moe_ffn")
        return self.bufs["y"], self.bufs["h"]

    def ffn_gate_up(self, stream=None, x=None):
        if self.fused_gather:
            _check(self._lib.brownout_moe_ffn_gate_up_gather(*self._fused_args(self._gate_up_args, x),
                                                             self._s(stream)), "brownout_moe_ffn_gate_up_gather")
        else:
            _check(self._lib.brownout_moe_ffn_gate_up(*self._gate_up_args, self._s(stream)),
                   "brownout_moe_ffn_gate_up")
        return self.bufs["h"]

    def ffn_down(self, stream=None):
        _check(self._lib.brownout_moe_ffn_down(*self._down_args, self._s(stream)), "brownout_moe_ffn_down")
        return self.bufs["y"]

    def shared(self, x, stream=None):
        self._x(x)  # the shared experts read x in token order: the layer's own input
        a = self._shared_args
        _check(self._lib.brownout_moe_ffn(*a[:6], x.data_ptr(), *a[6:], self._s(stream)), "brownout_moe_ffn")
        return self.bufs["y_sh"], self.bufs["h_sh"]

    def shared_fork(self, x, stream=None):
        """Starts the shared experts on the layer's side stream, after the work
        queued so far on `stream` (x is ready): they read only x, so they run
        beside route, dispatch and the routed FFN and fill the CUs those leave
        idle (the persistent GEMMs' partial last rounds, the short kernels).
        shared_join must follow before y_sh is read. Without a side stream
        (concurrent_shared=False or no shared experts) this is `shared`."""
        if self._side is None:
            return self.shared(x, stream)
        self._x(x)
        self._side.wait_stream(stream if stream is not None else torch.cuda.current_stream())
        a = self._shared_side_args
        _check(self._lib.brownout_moe_ffn(*a[:6], x.data_ptr(), *a[6:], self._side.cuda_stream),
               "brownout_moe_ffn")
        return self.bufs["y_sh"], self.bufs["h_sh"]

    def shared_join(self, stream=None):
        """Makes `stream` wait for the shared experts started by shared_fork."""
        if self._side is not None:
            (stream if stream is not None else torch.cuda.current_stream()).wait_stream(self._side)

    def combine(self, stream=None):
        _check(self._lib.brownout_moe_combine(self._desc_ref, *self._combine_args, self._s(stream)),
               "brownout_moe_combine")
        return self.bufs["out"]

    def down_combine(self, stream=None):
        """The down projection with the combine folded in (fold_combine layers)."""
        _check(self._lib.brownout_moe_ffn_down_combine(self._desc_ref, *self._down_combine_args, self._s(stream)),
               "brownout_moe_ffn_down_combine")
        return self.bufs["out"]

    def __call__(self, x: torch.Tensor, stream=None) -> torch.Tensor:
        shared = bool(self.desc.d_ff_shared)
        if shared:
            self.shared_fork(x, stream)
        self.route(x, stream)
        self.dispatch(x, stream)
        if self.fold_combine:
            self.ffn_gate_up(stream, x=x)
            if shared:
                self.shared_join(stream)
            return self.down_combine(stream)
        self.ffn(stream, x=x)
        if shared:
            self.shared_join(stream)
        return self.combine(stream)
