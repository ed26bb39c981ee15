"""The C ABI on the host (no GPU): the library loads, exports every function
the public header declares, and rejects bad arguments before any HIP call.
Every call here fails host validation (or is the T == 0 no-op), so nothing is
ever enqueued."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2607_04164_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "brownout_moe.h")

OK, NULL, SHAPE, ALIGN, MAP, UNSUP, WS = 0, 1, 2, 3, 4, 5, 6
FAKE = ctypes.c_void_p(0x10000)      # aligned, never dereferenced
MISALIGNED = ctypes.c_void_p(0x10008)


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"BMOE_API\s+[\w\s\*]+?\b(\w+)\s*\(", text)))


def test_header_constants_match_binding():
    text = open(HEADER).read()
    m = re.search(r"#define BMOE_DISPATCH_SCRATCH_BYTES (\d+)", text)
    assert m and int(m.group(1)) == B.DISPATCH_SCRATCH_BYTES
    m = re.search(r"#define BMOE_DISTILL_WS_BYTES (\d+)", text)
    assert m and int(m.group(1)) == B.DISTILL_WS_BYTES
    m = re.search(r"#define BMOE_ROUTE_RECHECK_GAP \(1\.0f / (\d+)\.0f\)", text)
    assert m and 1.0 / int(m.group(1)) == B.ROUTE_RECHECK_GAP


def good_desc(**kw):
    d = B.make_desc(T=64, d=256, E=8, top_k=2, G=4, d_ff=512, dtype="bf16")
    return d.replace(**kw) if kw else d


@pytest.fixture(scope="module")
def lib():
    return B.load_library()


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert len(names) >= 11, names
    for n in names:
        assert hasattr(lib, n), f"{n} declared in the header but not exported"
    assert set(names) == set(B.EXPORTED)


def test_version_and_status_strings(lib):
    assert lib.bmoe_version() == 10000
    for s in range(8):
        assert len(B.status_str(s)) >= 2


@pytest.mark.parametrize("field,value,code", [
    ("T", -1, SHAPE), ("E", 0, SHAPE), ("E", 257, SHAPE), ("top_k", 0, SHAPE), ("top_k", 9, SHAPE),
    ("G", 0, SHAPE), ("G", 9, SHAPE), ("d", 12, SHAPE), ("d", 0, SHAPE), ("d_ff", 20, SHAPE),
    ("d_ff_shared", 4, SHAPE), ("d_ff_shared", -8, SHAPE), ("norm_topk", 2, SHAPE), ("dtype", 3, UNSUP),
])
def test_validate_rejects(field, value, code):
    assert B.validate(good_desc(**{field: value})) == code


def test_validate_accepts_configs():
    from paper_2607_04164_amd import workload as W
    for cfg in W.CONFIGS.values():
        d = B.make_desc(cfg.T, cfg.d, cfg.E, cfg.top_k, cfg.G, cfg.d_ff, cfg.d_ff_shared,
                        cfg.norm_topk, cfg.dtype)
        assert B.validate(d) == OK, cfg.name
    assert B.validate(good_desc(E=256, top_k=16, G=256)) == OK
    assert B.validate(good_desc(top_k=17, E=64)) == SHAPE


def test_validate_map():
    assert B.validate_map([0, 1, 2, 3, 0, 1, 2, 3], 8, 4) == OK
    assert B.validate_map([0, 1, 2, 4, 0, 1, 2, 3], 8, 4) == MAP
    assert B.validate_map([0, -1, 2, 3, 0, 1, 2, 3], 8, 4) == MAP
    assert B.validate_map([0, 0], 2, 3) == SHAPE


def test_workspace_bytes():
    d = good_desc(T=1000, E=16, G=16)
    n = B.workspace_bytes(d, B.STAGE_DISPATCH)
    assert n == 256 + 4 * 16 * 8  # header + ceil(1000/256) tiles x G status words
    for st in (B.STAGE_ROUTE, B.STAGE_COMBINE):
        assert B.workspace_bytes(d, st) == 0
    # FFN: two fp32 256x256 accumulator tiles per CU of the current device (none
    # without a device, and none for fp32 layers)
    n = B.workspace_bytes(d, B.STAGE_FFN)
    assert n % (2 * 256 * 256 * 4) == 0
    assert B.workspace_bytes(d.replace(dtype=0), B.STAGE_FFN) == 0
    assert B.workspace_bytes(good_desc(E=0), B.STAGE_DISPATCH) == 0


def test_entry_points_reject_before_launch(lib):
    d = good_desc()
    bd = ctypes.byref(d)
    z = None
    # route
    assert lib.brownout_moe_route(bd, z, FAKE, z, z, FAKE, FAKE, FAKE, FAKE, FAKE, z, z) == NULL
    assert lib.brownout_moe_route(bd, FAKE, FAKE, z, z, z, FAKE, FAKE, FAKE, FAKE, z, z) == NULL
    assert lib.brownout_moe_route(bd, MISALIGNED, FAKE, z, z, FAKE, FAKE, FAKE, FAKE, FAKE, z, z) == ALIGN
    bad = ctypes.byref(good_desc(top_k=0))
    assert lib.brownout_moe_route(bad, FAKE, FAKE, z, z, FAKE, FAKE, FAKE, FAKE, FAKE, z, z) == SHAPE
    # dispatch
    need = B.workspace_bytes(d, B.STAGE_DISPATCH)
    assert lib.brownout_moe_dispatch(bd, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, z, need, z) == WS
    assert lib.brownout_moe_dispatch(bd, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, need - 1, z) == WS
    assert lib.brownout_moe_dispatch(bd, FAKE, MISALIGNED, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, need, z) == ALIGN
    assert lib.brownout_moe_dispatch(bd, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                                     ctypes.c_void_p(0x10010), need, z) == ALIGN
    assert lib.brownout_moe_dispatch(bd, z, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, need, z) == NULL
    # dispatch without row copies (x_perm NULL): x may be NULL; with x_perm, x may not
    assert lib.brownout_moe_dispatch(bd, FAKE, z, FAKE, FAKE, FAKE, FAKE, z, z, need, z) == WS
    assert lib.brownout_moe_dispatch(bd, FAKE, z, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, need, z) == NULL
    assert lib.brownout_moe_dispatch(bd, FAKE, z, z, FAKE, FAKE, FAKE, z, FAKE, need, z) == NULL
    # allocation-free dispatch: the same checks, and shapes beyond its array
    nd = lib.brownout_moe_dispatch_noalloc
    assert nd(bd, z, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, z) == NULL
    assert nd(bd, FAKE, MISALIGNED, FAKE, FAKE, FAKE, FAKE, FAKE, z) == ALIGN
    huge = good_desc(T=140000, E=256, G=256)
    assert B.workspace_bytes(huge, B.STAGE_DISPATCH) > B.DISPATCH_SCRATCH_BYTES
    assert nd(ctypes.byref(huge), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, z) == WS
    # ffn (and its halves)
    ffn = lib.brownout_moe_ffn
    assert ffn(9, 4, 128, 256, 512, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, z, 0, z) == UNSUP
    assert ffn(1, 0, 128, 256, 512, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, z, 0, z) == SHAPE
    assert ffn(1, 257, 128, 256, 512, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, z, 0, z) == SHAPE
    assert ffn(1, 4, 128, 250, 512, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, z, 0, z) == SHAPE
    assert ffn(1, 4, 128, 256, 512, z, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, z, 0, z) == NULL
    assert ffn(1, 4, 128, 256, 512, FAKE, FAKE, FAKE, FAKE, FAKE, MISALIGNED, FAKE, z, 0, z) == ALIGN
    # the stream-K workspace must be 256-byte aligned
    assert ffn(1, 4, 128, 256, 512, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, ctypes.c_void_p(0x10010), 1 << 30,
               z) == ALIGN
    # explicit stream-K threshold: -1 (default) .. 2^20
    fx = lib.brownout_moe_ffn_ex
    assert fx(1, 4, 128, 256, 512, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, z, 0, -2, z) == SHAPE
    assert fx(1, 4, 128, 256, 512, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, z, 0, (1 << 20) + 1, z) == SHAPE
    assert fx(1, 4, 128, 256, 512, z, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, z, 0, 0, z) == NULL
    assert fx(1, 4, 0, 256, 512, z, z, z, z, z, z, z, z, 0, 0, z) == OK
    assert lib.brownout_moe_ffn_gate_up(1, 4, 128, 256, 512, FAKE, z, FAKE, FAKE, FAKE, z, 0, z) == NULL
    assert lib.brownout_moe_ffn_down(1, 4, 128, 256, 512, FAKE, FAKE, FAKE, MISALIGNED, z, 0, z) == ALIGN
    # fused gather: row indices required, the source small enough for 32-bit offsets
    g = lib.brownout_moe_ffn_gather
    assert g(1, 4, 128, 256, 512, FAKE, z, 64, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, z, 0, z) == NULL
    assert g(1, 4, 128, 256, 512, FAKE, FAKE, 0, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, z, 0, z) == SHAPE
    assert g(1, 4, 128, 4096, 512, FAKE, FAKE, 1 << 19, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, z, 0, z) == SHAPE
    assert g(1, 4, 128, 256, 512, FAKE, FAKE, 64, MISALIGNED, FAKE, FAKE, FAKE, FAKE, FAKE, z, 0, z) == ALIGN
    assert g(1, 0, 128, 256, 512, FAKE, FAKE, 64, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, z, 0, z) == SHAPE
    gu = lib.brownout_moe_ffn_gate_up_gather
    assert gu(1, 4, 128, 256, 512, FAKE, z, 64, FAKE, FAKE, FAKE, FAKE, z, 0, z) == NULL
    assert gu(1, 4, 128, 256, 512, FAKE, FAKE, 64, FAKE, FAKE, z, FAKE, z, 0, z) == NULL
    # grouping search
    ui = lib.brownout_moe_united_init
    assert ui(9, 8, 4, 256, 512, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, z) == UNSUP
    assert ui(1, 0, 4, 256, 512, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, z) == SHAPE
    assert ui(1, 8, 257, 256, 512, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, z) == SHAPE
    assert ui(1, 8, 4, 250, 512, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, z) == SHAPE
    assert ui(1, 8, 4, 256, 512, z, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, z) == NULL
    assert ui(1, 8, 4, 256, 512, FAKE, FAKE, FAKE, FAKE, FAKE, MISALIGNED, FAKE, z) == ALIGN
    dm = lib.brownout_moe_distill_mse
    W = B.DISTILL_WS_BYTES
    assert dm(9, 8, 4, 100, 256, FAKE, FAKE, FAKE, FAKE, FAKE, z, FAKE, W, z) == UNSUP
    assert dm(1, 8, 4, -1, 256, FAKE, FAKE, FAKE, FAKE, FAKE, z, FAKE, W, z) == SHAPE
    assert dm(1, 8, 4, 100, 260, FAKE, FAKE, FAKE, FAKE, FAKE, z, FAKE, W, z) == SHAPE
    assert dm(1, 8, 4, 100, 256, FAKE, z, FAKE, FAKE, FAKE, z, FAKE, W, z) == NULL
    assert dm(1, 8, 4, 100, 256, FAKE, FAKE, MISALIGNED, FAKE, FAKE, z, FAKE, W, z) == ALIGN
    assert dm(1, 8, 4, 100, 256, FAKE, FAKE, FAKE, FAKE, FAKE, z, z, W, z) == WS
    assert dm(1, 8, 4, 100, 256, FAKE, FAKE, FAKE, FAKE, FAKE, z, FAKE, 64, z) == WS
    assert dm(1, 8, 4, 0, 256, z, z, z, z, z, z, z, 0, z) == OK
    # combine
    assert lib.brownout_moe_combine(bd, FAKE, FAKE, FAKE, z, z, z) == NULL
    assert lib.brownout_moe_combine(bd, FAKE, FAKE, FAKE, MISALIGNED, FAKE, z) == ALIGN


def test_zero_tokens_needs_no_pointers(lib):
    d = good_desc(T=0)
    bd = ctypes.byref(d)
    z = None
    assert lib.brownout_moe_route(bd, z, z, z, z, z, z, z, z, z, z, z) == OK
    assert lib.brownout_moe_dispatch(bd, z, z, z, z, z, z, z, z, 0, z) == OK
    assert lib.brownout_moe_dispatch_noalloc(bd, z, z, z, z, z, z, z, z) == OK
    assert lib.brownout_moe_combine(bd, z, z, z, z, z, z) == OK
    assert lib.brownout_moe_ffn(1, 4, 0, 256, 512, z, z, z, z, z, z, z, z, 0, z) == OK
    assert lib.brownout_moe_ffn_gather(1, 4, 0, 256, 512, z, z, 0, z, z, z, z, z, z, z, 0, z) == OK


def test_binding_refuses_host_tensors():
    import torch
    d = good_desc()
    with pytest.raises(ValueError):
        B.route(d, torch.zeros(64, 256), torch.zeros(8, 256), None, torch.zeros(8, dtype=torch.int32))


def test_missing_library_fails_loudly(tmp_path, monkeypatch):
    monkeypatch.setattr(B, "_lib", None)
    with pytest.raises(RuntimeError):
        B.load_library(str(tmp_path / "nope.so"))
