"""HIP path against the CPU oracle, through the C ABI (needs an MI355X).

Each stage is first fed the oracle's own upstream outputs, so a failure names
one stage; then the whole layer runs end to end. Small cases (the oracle runs
them in seconds) span several route/dispatch/FFN tiles and end in ragged
tails; the full-size workloads are checked in full on every integer output
and on a sample of tokens (including the first and last row of every group)
for the float outputs, since each token's output depends on that token only.
"""
from __future__ import annotations

import dataclasses
import functools

import numpy as np
import pytest
import torch

import oracle
from oracle.partial import partial_map
from gpu_util import (TOL, assert_close_rows, assert_gates, desc_of, dev_tensor, device_weights,
                      group_boundary_tokens, host_f32, stream_k_split_rows, to_storage)
from paper_2607_04164_amd import binding as B
from paper_2607_04164_amd import brownout as BO
from paper_2607_04164_amd import workload as W

pytestmark = pytest.mark.gpu

SMALL = {
    "tiny": W.CONFIGS["tiny"],
    "mixtral-s": W.CONFIGS["mixtral"].with_(name="mixtral-s", T=300, d=512, d_ff=640),
    "fine-s": W.CONFIGS["fine"].with_(name="fine-s", T=517, d=256, d_ff=384),
    "heavy-s": W.CONFIGS["heavy"].with_(name="heavy-s", T=700, d=512, d_ff=192, d_ff_shared_each=192),
    "decode": W.CONFIGS["decode"],
    "tail": W.LayerConfig("tail", T=33, d=264, E=12, top_k=3, G=5, d_ff=520, dtype="bf16", zipf_s=1.2),
    # d_ff not a whole 64-column K-step: the register-staged 128-row tiles
    # (whole 64-column K-steps take the persistent 256-row kernel at any size)
    "ragged-s": W.CONFIGS["mixtral"].with_(name="ragged-s", T=300, d=520, d_ff=600),
}
CASES = [(n, 0) for n in SMALL] + [("tiny", 1), ("tiny", 2), ("fine-s", 1)]
IDS = [f"{n}-seed{s}" for n, s in CASES]


@functools.lru_cache(maxsize=None)
def case(name, seed):
    cfg = SMALL[name]
    L = W.make_layer(cfg, seed)
    ref = oracle.layer(L, want_intermediates=True)
    return L, ref


@pytest.fixture(scope="module", autouse=True)
def _lib():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load_library()


# ---------------------------------------------------------------------------
# route

@pytest.mark.parametrize("name,seed", CASES, ids=IDS)
def test_route_logits_in_exact(name, seed):
    """Selection, softmax, map and merge on given fp32 logits: integers exact."""
    L, ref = case(name, seed)
    cfg = L.cfg
    z32 = ref["logits"].astype(np.float32)
    want = oracle.route_from_logits(z32, L.e2g, cfg.top_k, cfg.norm_topk)
    e2g = torch.from_numpy(L.e2g).cuda()
    got = B.route(desc_of(cfg), None, None, None, e2g, logits_in=torch.from_numpy(z32).cuda())
    torch.cuda.synchronize()
    for k in ("topk_idx", "slot_group"):
        assert np.array_equal(got[k].cpu().numpy(), want[k]), k
    assert_gates(got["topk_w"].cpu().numpy(), want["topk_w"], "topk_w")
    assert_gates(got["slot_gate"].cpu().numpy(), want["slot_gate"], "slot_gate")


@pytest.mark.parametrize("name,seed", CASES, ids=IDS)
def test_route_exact(name, seed):
    """Logits computed on the GPU (MFMA for bf16): integers exact against float64 selection."""
    L, ref = case(name, seed)
    cfg = L.cfg
    w = device_weights(L)
    x = dev_tensor(L.x, cfg.dtype)
    got = B.route(desc_of(cfg), x, w["w_router"], w["bias"], w["e2g"], want_logits=True)
    torch.cuda.synchronize()
    zerr = np.abs(got["logits"].cpu().numpy().astype(np.float64) - ref["logits"]).max()
    # premise of the float64 recheck: fast logits are far closer than the gap
    assert zerr < B.ROUTE_RECHECK_GAP / 4, f"fp32 logit error {zerr:.3e}"
    for k in ("topk_idx", "slot_group"):
        assert np.array_equal(got[k].cpu().numpy(), ref[k]), k
    assert_gates(got["topk_w"].cpu().numpy(), ref["topk_w"], "topk_w")
    assert_gates(got["slot_gate"].cpu().numpy(), ref["slot_gate"], "slot_gate")


@pytest.mark.parametrize("E,d,k", [(16, 256, 4), (8, 256, 4), (8, 4096, 4), (16, 256, 10)],
                         ids=["ring-E16", "ring-E8", "direct-E8-d4096", "ring-E16-k10"])
def test_route_near_ties_decided_in_f64(E, d, k):
    """Two experts whose logits differ by far less than the fp32 rounding error
    (and exact ties) are still ordered as float64 orders them (on the LDS-ring
    logits path, on the direct path of routers with at most 8 experts, and with
    more picks than the register pick list holds)."""
    cfg = W.LayerConfig("ties", T=96, d=d, E=E, top_k=k, G=4, d_ff=64, dtype="bf16", zipf_s=1.0)
    L = W.make_layer(cfg, 5)
    # expert 7's router row equals expert 3's except one bf16 ulp in column 17;
    # column 17 of x is tiny, so the two logits differ by |x[t,17]| * ulp
    wr = L.w_router.copy()
    wr[7] = wr[3]
    wr[7, 17] = wr[3, 17] + 1
    L.w_router = wr
    x = W.bf16_bits_to_f32(L.x).copy()
    signs = np.where(np.arange(cfg.T) % 2 == 0, 1.0, -1.0)
    x[:, 17] = signs * 2.0 ** -(8 + np.arange(cfg.T) % 8)
    x[::12, 17] = 0.0  # exact ties: lower expert index first
    L.x = W.f32_to_bf16_bits(x.astype(np.float32))
    L.bias = L.bias.copy()
    L.bias[7] = L.bias[3] = np.float32(0.5)
    ref = oracle.route(L.f32("x"), L.f32("w_router"), L.bias, L.e2g, cfg.top_k)
    d37 = np.abs(ref["logits"][:, 3] - ref["logits"][:, 7])
    assert d37.max() < 1e-5 and (d37 == 0).any()
    w = device_weights(L)
    got = B.route(desc_of(cfg), dev_tensor(L.x, "bf16"), w["w_router"], w["bias"], w["e2g"])
    torch.cuda.synchronize()
    assert np.array_equal(got["topk_idx"].cpu().numpy(), ref["topk_idx"])
    assert np.array_equal(got["slot_group"].cpu().numpy(), ref["slot_group"])
    assert_gates(got["slot_gate"].cpu().numpy(), ref["slot_gate"], "slot_gate")


@pytest.mark.parametrize("E,d,k,T", [(8, 1024, 2, 300), (8, 2048, 2, 300), (8, 3072, 3, 257), (5, 4096, 2, 300),
                                     (3, 2048, 1, 40), (8, 4096, 8, 300), (16, 256, 9, 300), (16, 1024, 3, 300),
                                     (17, 512, 3, 4100), (33, 1024, 5, 4111), (64, 2048, 6, 8200),
                                     (60, 2048, 9, 4096)],
                         ids=["direct-d1024", "direct-d2048", "direct-d3072", "direct-E5", "direct-E3-k1",
                              "direct-k8", "ring-k9", "ring-E16-d1024", "xdirect-E17-d512", "xdirect-E33-d1024",
                              "xdirect-2perCU", "xdirect-k9"])
def test_route_shapes(E, d, k, T):
    """Every bf16 logits path and both pick lists (registers for k <= 8, LDS
    beyond) on ragged token counts: integers exact, gates to tolerance."""
    cfg = W.LayerConfig("rshape", T=T, d=d, E=E, top_k=k, G=max(1, E // 2), d_ff=64, dtype="bf16", zipf_s=1.0,
                        norm_topk=1 if k == 2 else 0)
    L = W.make_layer(cfg, 3, with_weights=False)
    ref = oracle.route(L.f32("x"), L.f32("w_router"), L.bias, L.e2g, cfg.top_k, cfg.norm_topk)
    w = {"w_router": dev_tensor(L.w_router, "bf16"), "bias": torch.from_numpy(L.bias).cuda(),
         "e2g": torch.from_numpy(L.e2g).cuda()}
    got = B.route(desc_of(cfg), dev_tensor(L.x, "bf16"), w["w_router"], w["bias"], w["e2g"], want_logits=True)
    torch.cuda.synchronize()
    zerr = np.abs(got["logits"].cpu().numpy().astype(np.float64) - ref["logits"]).max()
    assert zerr < B.ROUTE_RECHECK_GAP / 4, f"fp32 logit error {zerr:.3e}"
    for key in ("topk_idx", "slot_group"):
        assert np.array_equal(got[key].cpu().numpy(), ref[key]), key
    assert_gates(got["topk_w"].cpu().numpy(), ref["topk_w"], "topk_w")
    assert_gates(got["slot_gate"].cpu().numpy(), ref["slot_gate"], "slot_gate")


# ---------------------------------------------------------------------------
# dispatch

@pytest.mark.parametrize("name,seed", CASES, ids=IDS)
def test_dispatch_exact(name, seed):
    L, ref = case(name, seed)
    cfg = L.cfg
    desc = desc_of(cfg)
    sg = torch.from_numpy(ref["slot_group"]).cuda()
    x = dev_tensor(L.x, cfg.dtype)
    ws = B.new_dispatch_workspace(desc, "cuda")
    got = B.dispatch(desc, sg, x, ws)
    torch.cuda.synchronize()
    N = ref["N"]
    assert np.array_equal(got["counts"].cpu().numpy(), ref["counts"])
    assert np.array_equal(got["offsets"].cpu().numpy(), ref["offsets"])
    assert np.array_equal(got["perm_token"][:N].cpu().numpy(), ref["perm_token"])
    assert np.array_equal(got["slot_row"].cpu().numpy(), ref["slot_row"])
    xp = got["x_perm"][:N]
    want = x[torch.from_numpy(ref["perm_token"]).long().cuda()]
    assert torch.equal(xp.view(torch.int16) if cfg.dtype == "bf16" else xp.view(torch.int32),
                       want.view(torch.int16) if cfg.dtype == "bf16" else want.view(torch.int32))
    assert int(ws.count_nonzero()) == 0, "dispatch must leave its workspace all zero"


@pytest.mark.parametrize("name", ["fine-s", "decode"], ids=["two-kernels", "one-tile"])
def test_dispatch_reports_a_dirty_workspace(name):
    """A workspace left with a stale tile ticket (as a call cut short between
    its two kernels would leave it): the call writes the "no rows" result
    with offsets[G] = -1 instead of stale or partial rows, leaves the
    workspace zero, and the next call is correct; on the histogram +
    permute path and on the one-kernel path of at most 256 tokens. Every
    kernel exits normally (the stale tickets are past the tile count)."""
    L, ref = case(name, 0)
    cfg = L.cfg
    desc = desc_of(cfg)
    sg = torch.from_numpy(ref["slot_group"]).cuda()
    x = dev_tensor(L.x, cfg.dtype)
    ws = B.new_dispatch_workspace(desc, "cuda")
    ntiles = -(-cfg.T // 256)
    ws.view(torch.int32)[0] = ntiles + 5  # stale ticket
    got = B.dispatch(desc, sg, x, ws)
    torch.cuda.synchronize()
    assert got["offsets"].cpu().numpy().tolist() == [0] * cfg.G + [-1]
    assert int(got["counts"].abs().sum()) == 0
    assert bool((got["slot_row"] == -1).all())
    assert int(ws.count_nonzero()) == 0
    got = B.dispatch(desc, sg, x, ws)
    torch.cuda.synchronize()
    assert np.array_equal(got["offsets"].cpu().numpy(), ref["offsets"])
    assert np.array_equal(got["slot_row"].cpu().numpy(), ref["slot_row"])
    for copy_rows in (False, True):  # the index-only kernel reports it the same way
        ws.view(torch.int32)[0] = ntiles
        got = B.dispatch(desc, sg, x if copy_rows else None, ws, copy_rows=copy_rows)
        torch.cuda.synchronize()
        assert int(got["offsets"][-1]) == -1 and bool((got["slot_row"] == -1).all())
        assert int(ws.count_nonzero()) == 0


def test_dispatch_many_tiles_and_reuse():
    """Several calls in a row on one workspace, T spanning many 256-token tiles.

    The group counts cover every width of the look-back's lane segments (64
    lanes per group for G <= 4 down to one lane for G = 256), and the longer
    runs need more than one look-back window per group.
    """
    r = np.random.default_rng(3)
    for T, k, G in ((5000, 6, 16), (777, 2, 4), (256, 4, 15), (1, 1, 1), (4097, 8, 64),
                    (40000, 2, 4), (30000, 3, 3), (17000, 5, 5), (9000, 4, 33), (3000, 8, 256)):
        sg = r.integers(-1, G, size=(T, k)).astype(np.int32)
        for t in range(T):  # at most one valid slot per group per token, as route guarantees
            seen = set()
            for i in range(k):
                if sg[t, i] in seen:
                    sg[t, i] = -1
                elif sg[t, i] >= 0:
                    seen.add(sg[t, i])
        ref = oracle.dispatch(sg, G)
        desc = B.make_desc(T, 64, max(G, k), k, G, 64)
        x = torch.randn(T, 64, device="cuda").to(torch.bfloat16)
        ws = B.new_dispatch_workspace(B.make_desc(40000, 64, 256, 8, 256, 64), "cuda")
        for _ in range(2):
            got = B.dispatch(desc, torch.from_numpy(sg).cuda(), x, ws)
            torch.cuda.synchronize()
            assert np.array_equal(got["offsets"].cpu().numpy(), ref["offsets"])
            assert np.array_equal(got["slot_row"].cpu().numpy(), ref["slot_row"])
            assert np.array_equal(got["perm_token"][:ref["N"]].cpu().numpy(), ref["perm_token"])
        assert int(ws.count_nonzero()) == 0


# ---------------------------------------------------------------------------
# ffn

@pytest.mark.parametrize("name,seed", CASES, ids=IDS)
def test_ffn(name, seed):
    L, ref = case(name, seed)
    cfg = L.cfg
    N, cap = ref["N"], cfg.T * cfg.top_k
    w = device_weights(L)
    a = torch.full((cap, cfg.d), 7.0, device="cuda", dtype=torch.bfloat16 if cfg.dtype == "bf16" else torch.float32)
    a[:N] = dev_tensor(to_storage(ref["x_perm"], cfg.dtype), cfg.dtype)
    sentinel = -3.0
    y = torch.full_like(a, sentinel)
    offs = torch.from_numpy(ref["offsets"]).cuda()
    yg, hg = B.ffn(offs, a, w["w_gate"], w["w_up"], w["w_down"], y=y)
    torch.cuda.synchronize()
    assert_close_rows(host_f32(hg[:N]), ref["h"], cfg.dtype, "h")
    assert_close_rows(host_f32(yg[:N]), ref["y"], cfg.dtype, "y")
    assert bool((yg[N:] == sentinel).all()), "rows past offsets[G] must not be written"
    if cfg.n_shared:
        xs = dev_tensor(L.x, cfg.dtype)
        ys, _ = B.ffn(torch.tensor([0, cfg.T], dtype=torch.int32, device="cuda"), xs, w["w_gate_sh"],
                      w["w_up_sh"], w["w_down_sh"])
        torch.cuda.synchronize()
        assert_close_rows(host_f32(ys), ref["y_shared"], cfg.dtype, "y_shared")


@pytest.mark.parametrize("spare", [5, 200], ids=["skinny", "tile128"])
def test_ffn_skewed_and_empty_segments(spare):
    """Hot/cold segment sizes (1 row .. many tiles) and empty segments anywhere.

    With 5 spare rows the capacity averages under 64 rows per segment, which
    selects the skinny kernels (the 300- and 129-row segments take several
    64-row passes); with 200 spare rows the 128-row tiles run.
    """
    r = np.random.default_rng(11)
    d, f, nseg = 256, 200, 7
    sizes = [0, 1, 300, 0, 129, 2, 0]
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    N = int(offsets[-1])
    a = W.f32_to_bf16_bits(r.standard_normal((N + spare, d)).astype(np.float32))
    wg = W.f32_to_bf16_bits((r.standard_normal((nseg, f, d)) / 16).astype(np.float32))
    wu = W.f32_to_bf16_bits((r.standard_normal((nseg, f, d)) / 16).astype(np.float32))
    wd = W.f32_to_bf16_bits((r.standard_normal((nseg, d, f)) / 16).astype(np.float32))
    ref_y = oracle.ffn(offsets, W.bf16_bits_to_f32(a), *(W.bf16_bits_to_f32(t) for t in (wg, wu, wd)))
    yg, _ = B.ffn(torch.from_numpy(offsets).cuda(), dev_tensor(a, "bf16"), dev_tensor(wg, "bf16"),
                  dev_tensor(wu, "bf16"), dev_tensor(wd, "bf16"))
    torch.cuda.synchronize()
    assert_close_rows(host_f32(yg[:N]), ref_y, "bf16", "y")


SKINNY_FFN = [
    # (segment sizes, spare rows, d, d_ff): capacity <= 64 rows per segment on
    # average selects the skinny kernels
    ((9, 14, 55, 59, 45, 32, 27, 62), 81, 2048, 1408),  # decode-shaped layer (G=8, top-6 of 64 tokens)
    ((3, 0, 70, 1), 2, 328, 136),     # K tails (328 = 256 + 72, 136), N tails (136 = 2*64 + 8), two passes
    ((64, 65, 1, 0, 120), 0, 264, 72),  # exact and ragged 64-row passes, 72 = 64 + 8 columns
    # K multiples of 64 select the all-copy kernels: fewer chunks than ring
    # slots (K = 64, 192, 320), N tails, two passes, empty segments
    ((3, 0, 70, 1), 2, 320, 192),
    ((64, 65, 1, 0, 120), 0, 136, 64),
]


@pytest.mark.parametrize("sizes,spare,d,f", SKINNY_FFN, ids=[f"seg{len(c[0])}-d{c[2]}-f{c[3]}" for c in SKINNY_FFN])
def test_ffn_skinny_paths(sizes, spare, d, f):
    """Decode-sized segments: skinny weight-streaming kernels against the oracle."""
    r = np.random.default_rng(len(sizes) * 1000 + d)
    nseg = len(sizes)
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    N = int(offsets[-1])
    cap = N + spare
    assert cap <= 64 * nseg
    a = W.f32_to_bf16_bits(r.standard_normal((cap, d)).astype(np.float32))
    wg = W.f32_to_bf16_bits((r.standard_normal((nseg, f, d)) / np.sqrt(d)).astype(np.float32))
    wu = W.f32_to_bf16_bits((r.standard_normal((nseg, f, d)) / np.sqrt(d)).astype(np.float32))
    wd = W.f32_to_bf16_bits((r.standard_normal((nseg, d, f)) / np.sqrt(f)).astype(np.float32))
    ref_y = oracle.ffn(offsets, W.bf16_bits_to_f32(a), *(W.bf16_bits_to_f32(t) for t in (wg, wu, wd)))
    yg, _ = B.ffn(torch.from_numpy(offsets).cuda(), dev_tensor(a, "bf16"), dev_tensor(wg, "bf16"),
                  dev_tensor(wu, "bf16"), dev_tensor(wd, "bf16"))
    torch.cuda.synchronize()
    assert_close_rows(host_f32(yg[:N]), ref_y, "bf16", "y")


# 60 segments of skewed sizes (1/rank), every seventh empty: ~200 rows per
# segment on average, the many small groups of an ungrouped layer
_SIZES60 = tuple(0 if i % 7 == 0 else 3000 // (i + 1) for i in range(60))

LARGE_TILE_FFN = [
    # (segment sizes, rows_cap, d, d_ff): above the skinny kernels' size, d and
    # d_ff multiples of 64 select the persistent direct-to-LDS kernel at any
    # group size; otherwise rows_cap >= 1024 * segments selects the register-
    # staged 256-row tiles
    ((700, 333), 2048, 256, 384),
    (_SIZES60, sum(_SIZES60) + 300, 256, 192),
    ((1000, 0, 513, 1), 4096, 320, 448),   # N tails in both GEMMs, empty and 1-row segments
    ((0, 1290), 2048, 512, 192),
    ((1000, 0, 513, 1), 4096, 288, 352),   # not multiples of 64: register-staged 256-row kernels
    ((257,), 1024, 264, 200),
    # one and two K-steps per tile (K = 64, 128): the K loops without a
    # copying step, and stream-K pieces of a single K-step
    ((1500, 700), 4096, 64, 128),
    ((900, 300), 2048, 128, 64),
]


def ffn_workspace():
    """The stream-K FFN workspace of the current device."""
    n = B.workspace_bytes(B.make_desc(1, 64, 1, 1, 1, 64, dtype="bf16"), B.STAGE_FFN)
    assert n > 0
    return torch.empty(n, dtype=torch.uint8, device="cuda")


@pytest.mark.parametrize("stream_k", [False, True], ids=["tile-per-wg", "stream-k"])
@pytest.mark.parametrize("sizes,cap,d,f", LARGE_TILE_FFN, ids=[f"seg{len(c[0])}-d{c[2]}-f{c[3]}" for c in LARGE_TILE_FFN])
def test_ffn_large_tile_paths(sizes, cap, d, f, stream_k):
    """256-row tiles; with the stream-K workspace (and the split threshold at
    zero) these small problems have fewer tiles than CUs, so every tile's K
    loop is cut into several pieces that meet in the workspace."""
    r = np.random.default_rng(len(sizes) * 1000 + d)
    nseg = len(sizes)
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    N = int(offsets[-1])
    a = W.f32_to_bf16_bits(r.standard_normal((cap, d)).astype(np.float32))
    wg = W.f32_to_bf16_bits((r.standard_normal((nseg, f, d)) / np.sqrt(d)).astype(np.float32))
    wu = W.f32_to_bf16_bits((r.standard_normal((nseg, f, d)) / np.sqrt(d)).astype(np.float32))
    wd = W.f32_to_bf16_bits((r.standard_normal((nseg, d, f)) / np.sqrt(d)).astype(np.float32))
    ref_y, ref_h = oracle.ffn(offsets, W.bf16_bits_to_f32(a)[:max(N, 1)],
                              *(W.bf16_bits_to_f32(t) for t in (wg, wu, wd)), want_h=True)
    y = torch.full((cap, d), -5.0, dtype=torch.bfloat16, device="cuda")
    ws = ffn_workspace() if stream_k else None
    if ws is not None:
        ws.fill_(0xFF)  # stale contents must not matter
    yg, hg = B.ffn(torch.from_numpy(offsets).cuda(), dev_tensor(a, "bf16"), dev_tensor(wg, "bf16"),
                   dev_tensor(wu, "bf16"), dev_tensor(wd, "bf16"), y=y, workspace=ws, split_min_idle=0)
    torch.cuda.synchronize()
    assert_close_rows(host_f32(hg[:N]), ref_h, "bf16", "h")
    assert_close_rows(host_f32(yg[:N]), ref_y, "bf16", "y")
    assert bool((yg[N:] == -5.0).all()), "rows past offsets[n_seg] must not be written"


def test_ffn_stream_k_full_rounds_and_reuse():
    """More tiles than two rounds of workgroups (full rounds, then the split
    remainder); the workspace is reused by a second, smaller call; results
    match the tile-per-workgroup path within bf16 rounding and are
    deterministic."""
    r = np.random.default_rng(77)
    d, f = 512, 1024
    # gate/up: 77 M-tiles x 8 N-tiles = 616 tiles (one whole round on 256 CUs,
    # then the split); down: 154 tiles (split only)
    sizes = (6000, 5000, 8000, 1)
    cap = 20480
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    N = int(offsets[-1])
    nseg = len(sizes)
    a = dev_tensor(W.f32_to_bf16_bits(r.standard_normal((cap, d)).astype(np.float32)), "bf16")
    wg = dev_tensor(W.f32_to_bf16_bits((r.standard_normal((nseg, f, d)) / np.sqrt(d)).astype(np.float32)), "bf16")
    wu = dev_tensor(W.f32_to_bf16_bits((r.standard_normal((nseg, f, d)) / np.sqrt(d)).astype(np.float32)), "bf16")
    wd = dev_tensor(W.f32_to_bf16_bits((r.standard_normal((nseg, d, f)) / np.sqrt(f)).astype(np.float32)), "bf16")
    offs = torch.from_numpy(offsets).cuda()
    ws = ffn_workspace()
    # split threshold 0: split whenever whole tiles leave CUs idle
    y0, h0 = B.ffn(offs, a, wg, wu, wd)
    y1, h1 = B.ffn(offs, a, wg, wu, wd, workspace=ws, split_min_idle=0)
    y2, h2 = B.ffn(offs, a, wg, wu, wd, workspace=ws, split_min_idle=0)
    torch.cuda.synchronize()
    # rows past offsets[n_seg] are never written (the buffers are uninitialised there)
    assert torch.equal(y1[:N].view(torch.int16), y2[:N].view(torch.int16))
    assert torch.equal(h1[:N].view(torch.int16), h2[:N].view(torch.int16))
    assert_close_rows(host_f32(h1[:N]), host_f32(h0[:N]), "bf16", "h")
    assert_close_rows(host_f32(y1[:N]), host_f32(y0[:N]), "bf16", "y")
    # spot rows against the oracle (first/last row of every segment)
    rows = sorted({int(o) for o in offsets[:-1]} | {int(o) - 1 for o in offsets[1:] if o > 0})
    rows = [q for q in rows if q < N]
    wg32, wu32, wd32 = host_f32(wg), host_f32(wu), host_f32(wd)
    one = np.array([0, 1], np.int32)
    for q in rows:
        sg = int(np.searchsorted(offsets, q, side="right") - 1)
        ref_y, ref_h = oracle.ffn(one, host_f32(a[q:q + 1]), wg32[sg:sg + 1], wu32[sg:sg + 1], wd32[sg:sg + 1],
                                  want_h=True)
        assert_close_rows(host_f32(h1[q:q + 1]), ref_h, "bf16", f"h row {q} vs oracle")
        assert_close_rows(host_f32(y1[q:q + 1]), ref_y, "bf16", f"y row {q} vs oracle")
    # a smaller problem through the same (now stale) workspace
    small = np.array([0, 700, 1500], np.int32)
    ys, hs = B.ffn(torch.from_numpy(small).cuda(), a, wg[:2].contiguous(), wu[:2].contiguous(), wd[:2].contiguous(),
                   workspace=ws, split_min_idle=0)
    ys0, _ = B.ffn(torch.from_numpy(small).cuda(), a, wg[:2].contiguous(), wu[:2].contiguous(), wd[:2].contiguous())
    torch.cuda.synchronize()
    assert_close_rows(host_f32(ys[:1500]), host_f32(ys0[:1500]), "bf16", "y small")


# ---------------------------------------------------------------------------
# combine

@pytest.mark.parametrize("name,seed", CASES, ids=IDS)
def test_combine(name, seed):
    L, ref = case(name, seed)
    cfg = L.cfg
    cap = cfg.T * cfg.top_k
    y_store = to_storage(ref["y"], cfg.dtype)
    y = torch.zeros((cap, cfg.d), device="cuda", dtype=torch.bfloat16 if cfg.dtype == "bf16" else torch.float32)
    y[:ref["N"]] = dev_tensor(y_store, cfg.dtype)
    ysh_np = ysh = None
    if cfg.n_shared:
        ysh_np = to_storage(ref["y_shared"], cfg.dtype)
        ysh = dev_tensor(ysh_np, cfg.dtype)
    out = B.combine(desc_of(cfg), torch.from_numpy(ref["slot_row"]).cuda(),
                    torch.from_numpy(ref["slot_gate"]).cuda(), y, ysh)
    torch.cuda.synchronize()
    widen = (lambda a: W.bf16_bits_to_f32(a)) if cfg.dtype == "bf16" else (lambda a: a)
    want = oracle.combine(ref["slot_row"], ref["slot_gate"], widen(y_store),
                          None if ysh_np is None else widen(ysh_np), d=cfg.d)
    assert_close_rows(host_f32(out), want, cfg.dtype, "out")


# ---------------------------------------------------------------------------
# whole layer

def run_layer(L):
    cfg = L.cfg
    layer = B.LayerForward(desc_of(cfg), device_weights(L))
    out = layer(dev_tensor(L.x, cfg.dtype))
    torch.cuda.synchronize()
    return layer, out


def check_layer(L, ref, layer, out):
    cfg = L.cfg
    r, dsp = layer.bufs["route"], layer.bufs["dispatch"]
    for k in ("topk_idx", "slot_group"):
        assert np.array_equal(r[k].cpu().numpy(), ref[k]), k
    for k in ("counts", "offsets", "slot_row"):
        assert np.array_equal(dsp[k].cpu().numpy(), ref[k]), k
    assert np.array_equal(dsp["perm_token"][:ref["N"]].cpu().numpy(), ref["perm_token"])
    assert_gates(r["slot_gate"].cpu().numpy(), ref["slot_gate"], "slot_gate")
    assert_close_rows(host_f32(out), ref["out"], cfg.dtype, "out")


@pytest.mark.parametrize("name,seed", CASES, ids=IDS)
def test_layer_end_to_end(name, seed):
    L, ref = case(name, seed)
    layer, out = run_layer(L)
    check_layer(L, ref, layer, out)


EDGE = {
    "T1": W.LayerConfig("T1", T=1, d=128, E=8, top_k=2, G=4, d_ff=64, dtype="bf16", zipf_s=1.0),
    "k1": W.LayerConfig("k1", T=200, d=128, E=8, top_k=1, G=4, d_ff=96, dtype="bf16", zipf_s=1.0),
    "G1": W.LayerConfig("G1", T=150, d=128, E=16, top_k=4, G=1, d_ff=96, dtype="bf16", zipf_s=1.0),
    "identity": W.LayerConfig("identity", T=150, d=128, E=8, top_k=2, G=8, d_ff=96, dtype="bf16", zipf_s=1.0),
    "E1": W.LayerConfig("E1", T=70, d=64, E=1, top_k=1, G=1, d_ff=64, dtype="bf16", zipf_s=1.0),
    "maxE": W.LayerConfig("maxE", T=90, d=128, E=256, top_k=16, G=64, d_ff=64, dtype="bf16", zipf_s=1.1),
    "E100": W.LayerConfig("E100", T=300, d=192, E=100, top_k=5, G=20, d_ff=72, dtype="bf16", zipf_s=1.2),
    "k_eq_E": W.LayerConfig("k_eq_E", T=64, d=64, E=4, top_k=4, G=2, d_ff=64, dtype="bf16", zipf_s=1.0),
    "f32-tail": W.LayerConfig("f32-tail", T=45, d=72, E=10, top_k=3, G=4, d_ff=40, dtype="f32",
                              zipf_s=1.2, router_std=0.3, norm_topk=1),
}


@pytest.mark.parametrize("name", list(EDGE))
def test_layer_edge_shapes(name):
    cfg = EDGE[name]
    L = W.make_layer(cfg, 0)
    if name == "identity":
        L.e2g = np.arange(cfg.E, dtype=np.int32)
    ref = oracle.layer(L, want_intermediates=True)
    layer, out = run_layer(L)
    check_layer(L, ref, layer, out)


def test_layer_empty_groups_in_map():
    """Groups no expert maps to (first, middle and last) are legal and stay empty."""
    cfg = W.LayerConfig("holes", T=260, d=128, E=8, top_k=3, G=7, d_ff=64, dtype="bf16", zipf_s=1.0)
    L = W.make_layer(cfg, 2)
    L.e2g = np.array([1, 1, 2, 2, 4, 4, 5, 5], np.int32)
    ref = oracle.layer(L, want_intermediates=True)
    assert ref["counts"][0] == ref["counts"][3] == ref["counts"][6] == 0
    layer, out = run_layer(L)
    check_layer(L, ref, layer, out)


def test_zero_tokens_is_noop():
    cfg = W.LayerConfig("T0", T=0, d=64, E=8, top_k=2, G=4, d_ff=64, dtype="bf16", zipf_s=1.0)
    desc = desc_of(cfg)
    e = torch.zeros(8, dtype=torch.int32, device="cuda")
    x = torch.zeros((0, 64), dtype=torch.bfloat16, device="cuda")
    wr = torch.zeros((8, 64), dtype=torch.bfloat16, device="cuda")
    out = B.route(desc, x, wr, None, e)
    assert out["topk_idx"].shape == (0, 2)


def test_deterministic_bits():
    L, _ = case("heavy-s", 0)
    _, a = run_layer(L)
    _, b = run_layer(L)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


@pytest.mark.parametrize("name", ["heavy-s", "dma-shared"])
def test_shared_side_stream_bit_identical(name):
    """The shared experts on the layer's side stream (started once x is ready,
    joined before the combine) give the bits of the one-stream layer, call
    after call with no synchronisation between the forwards, also when the
    caller passes a stream of its own; y_sh equals the shared FFN run alone.
    (Neither shape splits a shared-FFN tile, so the one-stream layer's
    workspace changes no bit.)"""
    cfg = SMALL["heavy-s"] if name == "heavy-s" else FOLD["dma-shared"]
    L = W.make_layer(cfg, 3)
    w = device_weights(L)
    x = dev_tensor(L.x, cfg.dtype)
    one = B.LayerForward(desc_of(cfg), w, concurrent_shared=False)
    assert one._side is None
    want = one(x).clone()
    want_sh = one.bufs["y_sh"].clone()
    both = B.LayerForward(desc_of(cfg), w)
    assert both._side is not None
    outs = []
    for _ in range(3):
        outs.append(both(x).clone())
    caller = torch.cuda.Stream()
    caller.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(caller):
        outs.append(both(x, stream=caller).clone())
    torch.cuda.current_stream().wait_stream(caller)
    torch.cuda.synchronize()
    for i, o in enumerate(outs):
        assert torch.equal(o.view(torch.int16), want.view(torch.int16)), f"forward {i}"
    assert torch.equal(both.bufs["y_sh"], want_sh)
    check_layer(L, oracle.layer(L, want_intermediates=True), both, outs[-1])


def test_token_order_invariance():
    """Permuting tokens permutes the output rows bit for bit and keeps the counts."""
    L, _ = case("fine-s", 0)
    perm = np.random.default_rng(9).permutation(L.cfg.T)
    la, a = run_layer(L)
    L2 = dataclasses.replace(L, x=L.x[perm].copy())
    lb, b = run_layer(L2)
    assert torch.equal(b.view(torch.int16), a[torch.from_numpy(perm).long().cuda()].view(torch.int16))
    assert torch.equal(la.bufs["dispatch"]["counts"], lb.bufs["dispatch"]["counts"])


# ---------------------------------------------------------------------------
# full-size workloads: integers in full, floats on sampled tokens

def partial_layer(L):
    """The layer over the partial-brownout segment map of its threshold; the
    library's map builder must agree with the oracle's."""
    cfg = L.cfg
    e2s, seg = BO.segment_map(W.zipf_freq(L), L.e2g, cfg.G, cfg.theta)
    e2s_o, seg_o = partial_map(W.zipf_freq(L), L.e2g, cfg.G, cfg.theta)
    assert np.array_equal(e2s, e2s_o) and seg == seg_o
    return W.segment_layer(L, e2s, seg)


# ---------------------------------------------------------------------------
# fused gather: the FFN reads its rows from x through perm_token

GATHER = {
    "tiny": SMALL["tiny"],                     # fp32 kernels
    "mixtral-s": SMALL["mixtral-s"],           # persistent 256-row tiles, 150 rows per group
    "ragged-s": SMALL["ragged-s"],             # 128-row register-staged tiles
    "decode": SMALL["decode"],                 # skinny weight-streaming kernels
    "dma": W.LayerConfig("dma", T=2100, d=256, E=8, top_k=2, G=4, d_ff=384, dtype="bf16", zipf_s=0.5),
}


@pytest.mark.parametrize("name", list(GATHER))
@pytest.mark.parametrize("stream_k", [False, True], ids=["tiles", "stream_k"])
def test_ffn_gather_bit_identical(name, stream_k):
    """Dispatch without row copies + the gathering FFN writes the same bits as
    dispatch's x_perm + the FFN, on every kernel path; the permutation-only
    dispatch writes the same integers and leaves its workspace reusable."""
    cfg = GATHER[name]
    L = W.make_layer(cfg, 3)
    ref = oracle.route(L.f32("x"), L.f32("w_router"), L.bias, L.e2g, cfg.top_k, cfg.norm_topk)
    desc = desc_of(cfg)
    w = device_weights(L)
    x = dev_tensor(L.x, cfg.dtype)
    sg = torch.from_numpy(ref["slot_group"]).cuda()
    ws = B.new_dispatch_workspace(desc, "cuda")
    full = B.dispatch(desc, sg, x, ws)
    idx = B.dispatch(desc, sg, None, ws, copy_rows=False)
    idx2 = B.dispatch(desc, sg, x, ws, copy_rows=False)  # workspace left zero by the previous call
    torch.cuda.synchronize()
    N = int(full["offsets"][-1].item())
    for k in ("counts", "offsets", "slot_row"):
        assert torch.equal(idx[k], full[k]) and torch.equal(idx2[k], full[k]), k
    assert torch.equal(idx["perm_token"][:N], full["perm_token"][:N])
    assert "x_perm" not in idx
    fws = B.new_ffn_workspace(desc, "cuda") if stream_k else None
    y0, h0 = B.ffn(full["offsets"], full["x_perm"], w["w_gate"], w["w_up"], w["w_down"], workspace=fws)
    y1, h1 = B.ffn_gather(idx["offsets"], idx["perm_token"], x, w["w_gate"], w["w_up"], w["w_down"],
                          workspace=fws)
    h2 = B.ffn_gate_up_gather(idx["offsets"], idx["perm_token"], x, w["w_gate"], w["w_up"], workspace=fws)
    torch.cuda.synchronize()
    assert torch.equal(h1[:N], h0[:N]) and torch.equal(y1[:N], y0[:N])
    assert torch.equal(h2[:N], h0[:N])


@pytest.mark.parametrize("name", ["fine-s", "heavy-s", "tail"])
def test_layer_fused_gather(name):
    """The fused-gather layer: bit-identical to the four-call layer, and
    within tolerance of the oracle. The default layer takes the fused gather
    from top-3 on."""
    L, ref = case(name, 0)
    cfg = L.cfg
    w = device_weights(L)
    x = dev_tensor(L.x, cfg.dtype)
    assert B.LayerForward(desc_of(cfg), w).fused_gather == (cfg.top_k >= B.FUSED_GATHER_MIN_TOP_K)
    four = B.LayerForward(desc_of(cfg), w, fused_gather=False)
    assert "x_perm" in four.bufs["dispatch"]
    out0 = four(x).clone()
    layer = B.LayerForward(desc_of(cfg), w, fused_gather=True)
    out1 = layer(x)
    torch.cuda.synchronize()
    assert "x_perm" not in layer.bufs["dispatch"]
    assert torch.equal(out1, out0)
    check_layer(L, ref, layer, out1)


@pytest.mark.parametrize("name", ["mixtral", "fine", "heavy", "decode"])
def test_full_size_fused_gather_bit_identical(name):
    """At full size and with the stream-K workspace, the fused-gather layer
    writes the same bits as the four-call layer. test_full_size_sampled checks
    the default layer against the oracle (four calls at top-2, the fused
    gather from top-3 on), so this ties the other path to it."""
    L = full_case(name)
    cfg = L.cfg
    w = device_weights(L)
    x = dev_tensor(L.x, cfg.dtype)
    four = B.LayerForward(desc_of(cfg), w, fused_gather=False)
    assert "x_perm" in four.bufs["dispatch"]
    out0 = four(x).clone()
    layer = B.LayerForward(desc_of(cfg), w, fused_gather=True)
    out1 = layer(x)
    torch.cuda.synchronize()
    assert torch.equal(out1, out0)


# ---------------------------------------------------------------------------
# combine folded into the down projection's epilogue

FOLD = {
    # 256-row tiles with d a multiple of 128: the fold runs in the GEMM epilogue
    "dma": W.LayerConfig("dma", T=2100, d=256, E=8, top_k=2, G=4, d_ff=384, dtype="bf16", zipf_s=0.5),
    "dma-k1": W.LayerConfig("dma-k1", T=4500, d=384, E=8, top_k=1, G=4, d_ff=256, dtype="bf16", zipf_s=0.5),
    "dma-shared": W.LayerConfig("dma-shared", T=1200, d=256, E=16, top_k=6, G=4, d_ff=256, dtype="bf16",
                                zipf_s=1.5, n_shared=2, d_ff_shared_each=128),
    "mixtral-s": SMALL["mixtral-s"],  # the persistent kernel with 150 rows per group
    # other shapes: the down projection, then the combine kernel
    "ragged-s": SMALL["ragged-s"],
    "tiny": SMALL["tiny"],
}


@pytest.mark.parametrize("name", list(FOLD))
def test_layer_fold_combine(name):
    """The layer with the combine folded into the down projection: the same
    y and out bits as the unfused layer without the stream-K workspace (the
    fold never splits a tile), within tolerance of the oracle, on two calls
    in a row (the counter workspace is left zero)."""
    cfg = FOLD[name]
    L = W.make_layer(cfg, 4)
    ref = oracle.layer(L, want_intermediates=True)
    w = device_weights(L)
    x = dev_tensor(L.x, cfg.dtype)
    base = B.LayerForward(desc_of(cfg), w, stream_k=False)
    out0 = base(x).clone()
    y0 = base.bufs["y"].clone()
    fold = B.LayerForward(desc_of(cfg), w, fold_combine=True)
    for _ in range(2):
        fold.bufs["out"].fill_(7.0)
        out1 = fold(x)
        torch.cuda.synchronize()
        N = ref["N"]
        assert torch.equal(fold.bufs["y"][:N], y0[:N])
        assert torch.equal(out1, out0)
        assert int(fold.fold_ws.count_nonzero()) == 0, "the counters must be left zero"
    check_layer(L, ref, fold, out1)


# ---------------------------------------------------------------------------
# one GPU's share of a layer sharded over several GPUs

@pytest.mark.parametrize("base,P,r", [("mixtral-s", 8, 0), ("mixtral-s", 8, 7), ("heavy-s", 4, 2)])
def test_tp_share_layer(base, P, r):
    """Rank r's tensor-parallel share (d_ff/P hidden columns of every united
    and shared expert, route and dispatch replicated): its partial output
    against the oracle's partial output of the same share."""
    S = W.tp_share(W.make_layer(SMALL[base], 0), P, r)
    ref = oracle.layer(S, want_intermediates=True)
    layer, out = run_layer(S)
    check_layer(S, ref, layer, out)


@pytest.mark.parametrize("P", [2, 4, 16])
def test_ep_share_ffn(P):
    """Each rank's expert-parallel share: the grouped FFN over its block of
    united experts alone (offsets and weights from the block's first expert
    on) against the oracle on those rows, and no other row written; with 16
    ranks over 15 united experts one rank has none."""
    L, ref = case("fine-s", 0)
    cfg = L.cfg
    cap = cfg.T * cfg.top_k
    w = device_weights(L)
    a = torch.full((cap, cfg.d), 7.0, device="cuda", dtype=torch.bfloat16)
    a[:ref["N"]] = dev_tensor(to_storage(ref["x_perm"], cfg.dtype), cfg.dtype)
    offs = torch.from_numpy(ref["offsets"]).cuda()
    sentinel = -3.0
    for r in range(P):
        g0, g1 = W.ep_groups(cfg.G, P, r)
        if g0 == g1:
            continue
        lo, hi = int(ref["offsets"][g0]), int(ref["offsets"][g1])
        y = torch.full_like(a, sentinel)
        ys, hs = B.ffn(offs[g0:g1 + 1], a, w["w_gate"][g0:g1], w["w_up"][g0:g1], w["w_down"][g0:g1], y=y)
        torch.cuda.synchronize()
        assert_close_rows(host_f32(hs[lo:hi]), ref["h"][lo:hi], cfg.dtype, f"h rank {r}")
        assert_close_rows(host_f32(ys[lo:hi]), ref["y"][lo:hi], cfg.dtype, f"y rank {r}")
        assert bool((ys[:lo] == sentinel).all()) and bool((ys[hi:] == sentinel).all()), f"rank {r}"


def full_case(name):
    cfg = W.CONFIGS[name]
    L = W.make_layer(cfg, 0)
    return partial_layer(L) if cfg.theta is not None else L


@pytest.mark.parametrize("theta", [0.0, 0.6, 0.9, 1.0])
def test_partial_brownout_layer(theta):
    """Hot experts on their own FFN, cold ones on their united expert: the
    whole layer over the segment map (theta 0: full brownout, 1: zero
    brownout with all 60 original experts)."""
    cfg = W.CONFIGS["partial"].with_(name="partial-s", T=300, d=256, d_ff=192, theta=theta)
    PL = partial_layer(W.make_layer(cfg, 1))
    ref = oracle.layer(PL, want_intermediates=True)
    layer, out = run_layer(PL)
    check_layer(PL, ref, layer, out)


FULL_FLOAT_SAMPLE = {"mixtral": 1024, "heavy": 1024}  # tokens whose float outputs are checked


def _sample_tokens(cfg, dsp, n_random, seed):
    """Group-boundary tokens (first and last row of every segment), the first
    and last token, and n_random further tokens drawn without replacement."""
    rng = np.random.default_rng(seed)
    base = np.concatenate([group_boundary_tokens(dsp["perm_token"], dsp["offsets"]), [0, cfg.T - 1]])
    rest = np.setdiff1d(np.arange(cfg.T), base)
    extra = rng.choice(rest, size=min(n_random, rest.size), replace=False)
    return np.unique(np.concatenate([base, extra])).astype(np.int64)


def _check_full_size(L, layer, out, n_random, seed):
    """Integer outputs in full; float outputs (layer output and the united
    experts' rows) on a token sample against the oracle run on those tokens."""
    cfg = L.cfg
    r = oracle.route(L.f32("x"), L.f32("w_router"), L.bias, L.e2g, cfg.top_k, cfg.norm_topk)
    dsp = oracle.dispatch(r["slot_group"], cfg.G)
    gr, gd = layer.bufs["route"], layer.bufs["dispatch"]
    assert np.array_equal(gr["topk_idx"].cpu().numpy(), r["topk_idx"])
    assert np.array_equal(gr["slot_group"].cpu().numpy(), r["slot_group"])
    assert_gates(gr["slot_gate"].cpu().numpy(), r["slot_gate"], "slot_gate")
    for k in ("counts", "offsets", "slot_row"):
        assert np.array_equal(gd[k].cpu().numpy(), dsp[k]), k
    assert np.array_equal(gd["perm_token"][:dsp["N"]].cpu().numpy(), dsp["perm_token"])
    sample = _sample_tokens(cfg, dsp, n_random, seed)
    sub = dataclasses.replace(L, cfg=cfg.with_(T=len(sample)), x=L.x[sample].copy())
    ref = oracle.layer(sub, want_intermediates=True)
    assert np.array_equal(ref["topk_idx"], r["topk_idx"][sample])
    assert_close_rows(host_f32(out[torch.from_numpy(sample).cuda()]), ref["out"], cfg.dtype, "out")
    # united-expert outputs of the sampled tokens' rows
    sr = gd["slot_row"].cpu().numpy()[sample]
    rows = sr[sr >= 0]
    ref_rows = ref["slot_row"][sr >= 0]
    assert_close_rows(host_f32(layer.bufs["y"][torch.from_numpy(rows).long().cuda()]),
                      ref["y"][ref_rows], cfg.dtype, "y_perm")
    return r, dsp, sample


def _check_split_tiles(L, layer, dsp):
    """Every row of every output tile whose K loop the GEMMs split across
    workgroups (the stream-K pieces summed by the fixup kernel): h and y
    against the oracle's FFN on those rows."""
    cfg = L.cfg
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    offs = dsp["offsets"]
    rows_h = stream_k_split_rows(offs, cfg.d_ff, cfg.d, True, n_cu)
    rows_y = stream_k_split_rows(offs, cfg.d, cfg.d_ff, False, n_cu)
    rows = np.union1d(rows_h, rows_y).astype(np.int64)
    if rows.size == 0:
        return 0
    seg = np.searchsorted(offs, rows, side="right") - 1
    x = L.f32("x")
    wg, wu, wd = L.f32("w_gate"), L.f32("w_up"), L.f32("w_down")
    for s in np.unique(seg):
        rs = rows[seg == s]
        a = x[dsp["perm_token"][rs]]
        y_ref, h_ref = oracle.ffn(np.array([0, len(rs)], np.int32), a, wg[s:s + 1], wu[s:s + 1], wd[s:s + 1],
                                  want_h=True)
        idx = torch.from_numpy(rs).cuda()
        assert_close_rows(host_f32(layer.bufs["h"][idx]), h_ref, cfg.dtype, f"h split rows (segment {s})")
        assert_close_rows(host_f32(layer.bufs["y"][idx]), y_ref, cfg.dtype, f"y split rows (segment {s})")
    return rows.size


@pytest.mark.parametrize("name", ["decode", "fine", "heavy", "mixtral", "partial", "mixtral-tp8"])
def test_full_size_sampled(name):
    """Full-size workloads, seed 0, through LayerForward (the FFN with its
    stream-K workspace, as the benchmark runs it); mixtral-tp8 is rank 3's
    share of the Mixtral-shaped layer under 8-way tensor parallelism (d_ff
    1792). Integers in full; the float outputs of at least 1024 tokens at the
    Mixtral and heavy shapes (all of decode's 64), and every row of the tiles
    the GEMMs split."""
    L = W.tp_share(full_case("mixtral"), 8, 3) if name == "mixtral-tp8" else full_case(name)
    cfg = L.cfg
    layer, out = run_layer(L)
    _, dsp, sample = _check_full_size(L, layer, out, FULL_FLOAT_SAMPLE.get(name, 48), seed=1)
    if name in FULL_FLOAT_SAMPLE:
        assert len(sample) >= FULL_FLOAT_SAMPLE[name]
    n_split = _check_split_tiles(L, layer, dsp)
    if name == "mixtral":
        # the down GEMM's last partial round is split at this shape
        assert n_split > 0


@pytest.mark.parametrize("name", ["partial-theta1", "fine-ungrouped"])
def test_full_size_many_groups(name):
    """Full-size fine-grained layers with 60 small, skewed groups (about 530
    rows each on average): zero brownout over the segment map (theta 1, every
    expert on its own FFN) and the layer with G = E. They run the persistent
    256-row GEMM like the grouped layers; integers in full, floats sampled."""
    if name == "partial-theta1":
        L = partial_layer(W.make_layer(W.CONFIGS["partial"].with_(name="partial-theta1", theta=1.0), 0))
    else:
        cfg = W.CONFIGS["fine"]
        L = W.make_layer(cfg.with_(name="fine-ungrouped", G=cfg.E), 0)
    assert len(np.asarray(L.e2g).tolist()) == 60 and len(set(np.asarray(L.e2g).tolist())) == 60
    layer, out = run_layer(L)
    _, dsp, _ = _check_full_size(L, layer, out, 48, seed=3)
    _check_split_tiles(L, layer, dsp)


def test_full_size_fold_combine_bit_identical():
    """The Mixtral-shaped layer with the combine folded into the down
    projection writes the same out bits as the unfused layer without the
    stream-K workspace (whose parity with the oracle the sampled tests check)."""
    L = full_case("mixtral")
    cfg = L.cfg
    w = device_weights(L)
    x = dev_tensor(L.x, cfg.dtype)
    out0 = B.LayerForward(desc_of(cfg), w, stream_k=False)(x).clone()
    fold = B.LayerForward(desc_of(cfg), w, fold_combine=True)
    out1 = fold(x)
    torch.cuda.synchronize()
    assert torch.equal(out1, out0)
    assert int(fold.fold_ws.count_nonzero()) == 0


@pytest.mark.parametrize("seed", [1, 2])
@pytest.mark.parametrize("name", ["tiny", "decode", "fine", "heavy", "mixtral"])
def test_full_size_more_seeds(name, seed):
    """The five workloads at full size with seeds 1 and 2: every integer
    output in full, the float outputs on a sample of tokens."""
    L = W.make_layer(W.CONFIGS[name], seed)
    layer, out = run_layer(L)
    _check_full_size(L, layer, out, 32, seed=seed)
