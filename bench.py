"""Benchmark: grouped (full-brownout) MoE layer forward on one MI355X.

One step = one full layer forward over one batch of synthetic tokens, every
stage on the GPU: route (gate logits, softmax, top-k, expert-to-group map,
per-group merge) -> dispatch (group histogram, decoupled look-back scan,
row gather) -> FFN gate/up grouped GEMM -> FFN down grouped GEMM -> combine,
with the shared-expert FFN (layers that have one) on the layer's side stream
from the start of the step, joined before the combine. Inputs and weights are
resident in HBM before the timed region; nothing is allocated inside it.

Prints one JSON line. `value` is layer tokens/s over the K timed steps;
`roofline` is for the dominant kernel (the fused gate/up grouped GEMM) from
HIP events around its launches inside the timed steps (with shared experts,
from the per-stage pass, where it runs alone); `stages` gives every
stage's average time and achieved rate against its own roofline;
`cpu_baseline` times the CPU oracle on a bounded token sample.

    python bench.py [--steps K] [--warmup W] [--config mixtral|fine|heavy|decode|tiny]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA, TFLOP/s
VALU_F32_PEAK_TFLOPS = 157.3

# HBM bytes of one launch of the gate/up GEMM kernel, from rocprofv3 --pmc
# FETCH_SIZE and WRITE_SIZE runs of this bench (KiB per dispatch), scaled by
# what the same counters read for a plain 1 GiB device copy (bench.py
# --copy-probe-mib 1024: FETCH_SIZE reads half the copied bytes, WRITE_SIZE
# all of them). Valid only for the kernel sources they were taken with.
TRAFFIC_RECORDS = {
    "mixtral": {"src_sha1": "2efdf76e76bd4d124a9ba69e7eaa1ca11afd732e",
                "fetch_kib": 1524119.3, "write_kib": 217336.0, "fetch_scale": 2.0, "write_scale": 1.0,
                "profile": "profiles/gemm_gate_up_mixtral_hbm_counters.md"},
}
TRAFFIC_SOURCES = ("paper_2607_04164_amd/csrc/ffn.hip", "paper_2607_04164_amd/csrc/bmoe_common.h")


def recorded_traffic(config: str):
    """Scaled HBM bytes per launch of the dominant kernel, or None when no
    record exists or the kernel sources changed since it was taken."""
    import hashlib
    rec = TRAFFIC_RECORDS.get(config)
    if rec is None:
        return None
    h = hashlib.sha1()
    for f in TRAFFIC_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    if h.hexdigest() != rec["src_sha1"]:
        return None
    return int(rec["fetch_kib"] * 1024 * rec["fetch_scale"] + rec["write_kib"] * 1024 * rec["write_scale"])


WORKLOAD_TEXT = {
    "mixtral": "Mixtral-8x7B-shaped grouped MoE layer: T=4096 tokens, d=4096, E=8 experts, top-2, "
               "G=4 united experts (2 experts each, seeded map), SwiGLU d_ff=14336, bf16, "
               "router Zipf(s=1.0) skew",
    "fine": "fine-grained grouped MoE layer: T=8192, d=2048, E=60, top-4, G=15, d_ff=1408, bf16, Zipf(1.2)",
    "heavy": "heavy-skew grouped MoE layer: T=16384, d=2048, E=64 + 2 shared (1408 each), top-6, G=16, "
             "d_ff=1408, bf16, Zipf(1.5)",
    "decode": "decode-batch grouped MoE layer: T=64, d=2048, E=64, top-6, G=8, d_ff=1408, bf16, Zipf(1.2)",
    "tiny": "tiny fp32 grouped MoE layer: T=64, d=256, E=8, top-2, G=4, d_ff=512, Zipf(1.2)",
    "partial": "fine-grained MoE layer under partial brownout at threshold 0.4 (hot experts keep their own "
               "FFN, cold experts go to their united expert): T=8192, d=2048, E=60, top-4, G=15, d_ff=1408, "
               "bf16, Zipf(1.2)",
}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="mixtral", choices=sorted(WORKLOAD_TEXT))
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--share", default=None, metavar="tpP|epP",
                    help="one GPU's share of the layer sharded over P GPUs: tpP times rank --share-rank's "
                         "tensor-parallel slice (d_ff/P hidden columns; route and dispatch replicated); epP "
                         "also times each rank's grouped FFN over its block of united experts")
    ap.add_argument("--share-rank", type=int, default=0)
    ap.add_argument("--fused-gather", action="store_true",
                    help="time the fused-gather path as the headline: dispatch writes only the permutation and "
                         "the gate/up GEMM gathers its rows from x (no x_perm copy)")
    ap.add_argument("--distill", action="store_true",
                    help="instead of the layer forward: time the evaluation of one candidate grouping of the "
                         "workload's layer (parameter-average united experts, their FFN on the T tokens as "
                         "calibration set, the routing-weighted distillation errors)")
    ap.add_argument("--four-calls", action="store_true",
                    help="time the four-call path (dispatch writes x_perm) where the layer would take the fused "
                         "gather (top-3 and above)")
    ap.add_argument("--no-compare-fused", action="store_true",
                    help="skip the second timing of the same layer on the other gather path")
    ap.add_argument("--no-compare-fold", action="store_true",
                    help="skip timing the layer with the combine folded into the down projection")
    ap.add_argument("--theta", type=float, default=None,
                    help="partial-brownout threshold in [0, 1] (overrides the workload's; "
                         "0 is full brownout, 1 zero brownout)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="approximate CPU time budget of the oracle baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-graph", action="store_true",
                    help="skip timing the step captured into a HIP graph (graph_ms_per_step)")
    ap.add_argument("--no-compare-ungrouped", action="store_true",
                    help="skip timing the same layer with no grouping (G = E, every expert its own group: "
                         "zero brownout) and the speedup of grouping")
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the fine, heavy and decode workloads that the default (Mixtral-shaped) run "
                         "also times")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="instead of the layer: time a device-to-device copy of this many MiB (the plain "
                         "copy kernel that HBM byte counters are calibrated against)")
    return ap.parse_args()


def copy_probe(mib: int, reps: int = 10):
    """A plain device copy of a known size: reads and writes mib MiB per launch."""
    import torch
    n = mib * (1 << 20)
    src = torch.ones(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    print(json.dumps({"copy_probe_mib": mib, "bytes_read": n, "bytes_written": n, "launches": reps + 1,
                      "ms_per_copy": round(ms, 4), "GB_s_read_plus_write": round(2 * n / (ms * 1e-3) / 1e9, 1)}),
          flush=True)


_LAYERS = {}  # the last generated layer, reused when the same workload is timed again


def device_ffn_weights(cfg, seed, dev):
    """United-expert (and shared) FFN weights drawn on the device from the
    workload's distribution, N(0, 1/sqrt(d)) rounded to bf16: for timing-only
    runs (the extra workloads and the ungrouped comparison), where drawing
    gigabytes with numpy on the host would dominate the bench's run time."""
    import torch
    g = torch.Generator(device=dev)
    g.manual_seed(1_000_003 * seed + cfg.E * 131 + cfg.G)
    std = 1.0 / np.sqrt(cfg.d)

    def draw(shape):
        return (torch.randn(shape, generator=g, device=dev, dtype=torch.float32) * std).to(torch.bfloat16)

    G, f, d = cfg.G, cfg.d_ff, cfg.d
    w = {"w_gate": draw((G, f, d)), "w_up": draw((G, f, d)), "w_down": draw((G, d, f))}
    if cfg.n_shared:
        fs = cfg.d_ff_shared
        w.update(w_gate_sh=draw((1, fs, d)), w_up_sh=draw((1, fs, d)), w_down_sh=draw((1, d, fs)))
    return w


def graph_step_ms(step, reps):
    """Wall-clock ms per replay of one step captured into a HIP graph (None,
    with a note on stderr, if the capture fails)."""
    import torch
    try:
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step()
        g.replay()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(reps):
            g.replay()
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / reps
        del g
        return ms
    except RuntimeError as e:
        print(f"[bench] graph capture failed: {e}", file=sys.stderr, flush=True)
        torch.cuda.synchronize()
        return None


def time_layer(cfg, args, dev, device_weights=False):
    """Builds the seeded layer on the device and times args.steps full forwards
    after args.warmup untimed ones. Returns the host layer, the partial-brownout
    segment summary (or None), wall ms per step, the dominant kernel's event
    ms, per-stage event ms in the steps, alone and with cold caches, the row
    count N, the group row counts and the stages. device_weights: the FFN
    weights are drawn on the device (timing only; the route inputs still come
    from the seeded host generator)."""
    import torch
    from paper_2607_04164_amd import binding as B
    from paper_2607_04164_amd import workload as W

    key = (cfg, args.seed, device_weights)
    if key not in _LAYERS:
        print(f"[bench] generating {cfg.name} (G={cfg.G}) seed {args.seed}", file=sys.stderr, flush=True)
        _LAYERS.clear()
        _LAYERS[key] = W.make_layer(cfg, args.seed, with_weights=not device_weights)
    L0 = L = _LAYERS[key]
    seg_info = None
    if cfg.theta is not None:
        # partial brownout: the layer runs over the segment map (hot experts'
        # own FFNs, then united experts) built by the library's host code
        from paper_2607_04164_amd import brownout as BO
        e2s, seg = BO.segment_map(W.zipf_freq(L), L.e2g, cfg.G, cfg.theta)
        L = W.segment_layer(L, e2s, seg)
        cfg = L.cfg
        seg_info = {"theta": cfg.theta, "segments": len(seg),
                    "hot_experts": [i for kind, i in seg if kind == "expert"]}
    share = parse_share(args.share)
    if share and share[0] == "tp":
        L = W.tp_share(L, share[1], args.share_rank)
        cfg = L.cfg

    def to_dev(a):
        if cfg.dtype == "bf16":
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(a).to(dev)

    w = {"w_router": to_dev(L.w_router), "bias": torch.from_numpy(L.bias).to(dev),
         "e2g": torch.from_numpy(L.e2g).to(dev)}
    if device_weights:
        if cfg.theta is not None or cfg.dtype != "bf16":
            raise SystemExit("device-drawn weights are for the bf16 full-brownout workloads")
        w.update(device_ffn_weights(cfg, args.seed, dev))
    else:
        w.update(w_gate=to_dev(L.w_gate), w_up=to_dev(L.w_up), w_down=to_dev(L.w_down))
        if cfg.n_shared:
            w.update(w_gate_sh=to_dev(L.w_gate_sh), w_up_sh=to_dev(L.w_up_sh), w_down_sh=to_dev(L.w_down_sh))
    x = to_dev(L.x)
    desc = B.make_desc(cfg.T, cfg.d, cfg.E, cfg.top_k, cfg.G, cfg.d_ff, cfg.d_ff_shared, cfg.norm_topk,
                       cfg.dtype)
    # the layer's own choice of path unless asked for the fused gather (or the
    # x_perm rows an expert-parallel share needs)
    four_calls = getattr(args, "four_calls", False) or bool(share and share[0] == "ep")
    fused = True if getattr(args, "fused_gather", False) else (False if four_calls else None)
    fold = bool(getattr(args, "fold_combine", False))
    layer = B.LayerForward(desc, w, device=dev, fused_gather=fused, fold_combine=fold,
                           stream_k=not getattr(args, "no_stream_k", False))
    fused = layer.fused_gather

    if fold:
        # the shared experts' output feeds the folded combine
        stages = ["route", "dispatch", "ffn_gate_up"] + (["shared_ffn"] if cfg.n_shared else []) + ["down_combine"]
    else:
        stages = ["route", "dispatch", "ffn_gate_up", "ffn_down"] + (["shared_ffn"] if cfg.n_shared else []) + \
                 ["combine"]
    calls = {"route": lambda: layer.route(x), "dispatch": lambda: layer.dispatch(x),
             "ffn_gate_up": (lambda: layer.ffn_gate_up(x=x)) if fused else layer.ffn_gate_up,
             "ffn_down": layer.ffn_down,
             "shared_ffn": lambda: layer.shared(x), "combine": layer.combine,
             "down_combine": layer.down_combine if fold else None}

    # the layer's own schedule (LayerForward's order): with shared experts the
    # shared FFN starts on the layer's side stream first and joins before the
    # combine; the per-stage breakdown below runs the stages one after another
    # on one stream instead, so each is timed alone
    order = list(stages)
    if cfg.n_shared and layer._side is not None:
        order.remove("shared_ffn")
        order.insert(0, "shared_fork")
        order.insert(order.index("down_combine" if fold else "combine"), "shared_join")
    calls["shared_fork"] = lambda: layer.shared_fork(x)
    calls["shared_join"] = layer.shared_join

    def step(events=None):
        if events is None:
            for s in order:
                calls[s]()
            return
        for i, s in enumerate(stages):
            events[i].record()
            calls[s]()
        events[-1].record()

    dom_i = order.index("ffn_gate_up")

    def timed_step(e0, e1):
        # the headline steps: events only around the dominant kernel, so the
        # host work per step stays the library calls
        for i, s in enumerate(order):
            if i == dom_i:
                e0.record()
                calls[s]()
                e1.record()
            else:
                calls[s]()

    print(f"[bench] warmup {args.warmup}", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    N = int(layer.bufs["dispatch"]["offsets"][-1].item())
    counts = layer.bufs["dispatch"]["counts"].cpu().numpy().tolist()

    dev_ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    print(f"[bench] timing {args.steps} steps", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        timed_step(*dev_ev[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = wall * 1e3 / args.steps
    dom_ms = float(np.mean([a.elapsed_time(b) for a, b in dev_ev]))
    # per-stage breakdown: the same steps again with events around every stage
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(stages) + 1)] for _ in range(args.steps)]
    for k in range(args.steps):
        step(ev[k])
    torch.cuda.synchronize()
    per_stage_ms = {s: float(np.mean([ev[k][i].elapsed_time(ev[k][i + 1]) for k in range(args.steps)]))
                    for i, s in enumerate(stages)}
    if order != stages:
        # the timed steps ran the shared FFN beside the routed GEMMs, so their
        # events around the gate/up GEMM hold a shared GPU: its rate comes from
        # this pass, where it runs alone
        dom_ms = per_stage_ms["ffn_gate_up"]
    # the same step captured once into a HIP graph and replayed: the steps'
    # kernels without the host's launch work (wall clock over the replays)
    graph_ms = None
    if not getattr(args, "no_graph", False):
        graph_ms = graph_step_ms(step, args.steps)
    # each stage alone, launched back to back (the in-step events above also
    # hold the gaps between kernels, which dominate the short stages)
    iso_ms = {}
    for s in stages:
        reps = 3 if s.startswith("ffn") or s in ("shared_ffn", "down_combine") else 20
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        calls[s]()
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            calls[s]()
        e1.record()
        torch.cuda.synchronize()
        iso_ms[s] = e0.elapsed_time(e1) / reps
    # expert-parallel shares: each rank's grouped FFN over its block of united
    # experts, on the rows the whole dispatch gave that block
    ep_ms = None
    if share and share[0] == "ep":
        P = share[1]
        offs = layer.bufs["dispatch"]["offsets"]
        if fused:
            raise SystemExit("--share ep times the FFN on x_perm rows: run it without --fused-gather")
        a, h, y = layer.bufs["dispatch"]["x_perm"], layer.bufs["h"], layer.bufs["y"]
        ws = layer.ffn_ws
        ep_ms = []
        for r in range(P):
            g0, g1 = W.ep_groups(cfg.G, P, r)
            if g0 == g1:
                ep_ms.append(0.0)
                continue
            o = offs[g0:g1 + 1]
            wg, wu, wd = w["w_gate"][g0:g1], w["w_up"][g0:g1], w["w_down"][g0:g1]

            def ffn_r():
                B.ffn(o, a, wg, wu, wd, h=h, y=y, workspace=ws)
            ffn_r()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record()
            for _ in range(3):
                ffn_r()
            e1.record()
            torch.cuda.synchronize()
            ep_ms.append(e0.elapsed_time(e1) / 3)
    # every stage once more with cold caches: before each launch a read pass
    # over 1 GiB evicts L2 and the 256 MB MALL (a read, so no dirty lines are
    # left to be written back inside the timed launch)
    cold_ms = {}
    # float32, so that sum() is one reduction over the buffer (an integer sum
    # would first widen the whole buffer to int64, a 2 GiB write)
    flush = torch.ones(1 << 28, dtype=torch.float32, device=dev)
    for s in stages:
        reps = 3 if s.startswith("ffn") or s in ("shared_ffn", "down_combine") else 10
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        for e0, e1 in evs:
            flush.sum()
            e0.record()
            calls[s]()
            e1.record()
        torch.cuda.synchronize()
        cold_ms[s] = float(np.median([a.elapsed_time(b) for a, b in evs]))
    # the same protocol around a one-workgroup elementwise launch: the launch
    # and event overhead contained in every cold time above
    tiny = torch.zeros(64, device=dev)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(10)]
    for e0, e1 in evs:
        flush.sum()
        e0.record()
        tiny.add_(1.0)
        e1.record()
    torch.cuda.synchronize()
    cold_ms["launch_floor"] = float(np.median([a.elapsed_time(b) for a, b in evs]))
    del flush
    del layer, w, x
    torch.cuda.empty_cache()
    return L0, (cfg, seg_info, ep_ms, graph_ms, fused), ms_step, dom_ms, per_stage_ms, iso_ms, cold_ms, N, counts, \
        stages


def ungrouped_line(cfg, args, dev, ms_grouped):
    """The same layer with no grouping (G = E): tokens/s and the speedup of
    the grouped layer over it."""
    ucfg = cfg.with_(name=cfg.name + "-ungrouped", G=cfg.E, theta=None)
    uargs = argparse.Namespace(**{**vars(args), "share": None, "fused_gather": False})
    _, _, ms_u, _, _, iso_u, _, N_u, _, _ = time_layer(ucfg, uargs, dev, device_weights=True)
    return {"G": cfg.E, "rows_N": N_u, "value": round(cfg.T / (ms_u * 1e-3), 1), "ms_per_step": round(ms_u, 4),
            "stages_us": {k: round(v * 1e3, 2) for k, v in iso_u.items()},
            "grouped_speedup": round(ms_u / ms_grouped, 3),
            "note": "FFN weights drawn on the device (timing only)"}


def dominant_rate(cfg, N, counts, dom_ms, cold_ms):
    """The gate/up GEMM against its roofline: MFMA (4*N*d*d_ff flop, event
    time in the steps) or, for decode-sized batches on the weight-streaming
    kernel, HBM (weight bytes of the segments with rows, cold launch)."""
    T, d, k, f, s = cfg.T, cfg.d, cfg.top_k, cfg.d_ff, cfg.elem_bytes
    if T * k <= 64 * len(counts):
        S_w = sum(1 for c in counts if c > 0)
        by = 2 * S_w * d * f * s + N * d * s + N * f * s
        gbs = by / (cold_ms * 1e-3) / 1e9
        return {"kernel": "skinny_dma_kernel<gated>", "bound": "hbm", "us_cold": round(cold_ms * 1e3, 2),
                "GB_s": round(gbs, 1), "frac": round(gbs / HBM_PEAK_GBS, 4)}
    tf = 4.0 * N * d * f / (dom_ms * 1e-3) / 1e12
    return {"kernel": "grouped_gemm_dma_kernel<gated>", "bound": "mfma", "us": round(dom_ms * 1e3, 2),
            "TFLOP_s": round(tf, 1), "frac": round(tf / MFMA_BF16_PEAK_TFLOPS, 4)}


def parse_share(text):
    """"tp8" -> ("tp", 8), "ep4" -> ("ep", 4), None -> None."""
    if text is None:
        return None
    kind, num = text[:2], text[2:]
    if kind not in ("tp", "ep") or not num.isdigit() or int(num) < 1:
        raise SystemExit(f"--share must look like tp8 or ep4, got {text!r}")
    return kind, int(num)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs the layer on one GPU only; --gpus {args.gpus} is not supported "
              f"(the multi-GPU sharding is a design note, not part of this build)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2607_04164_amd import binding as B
    from paper_2607_04164_amd import workload as W

    if args.distill:
        torch.cuda.set_device(0)
        B.load_library()
        bench_distill(args, torch.device("cuda:0"))
        return

    if args.copy_probe_mib > 0:
        torch.cuda.set_device(0)
        copy_probe(args.copy_probe_mib)
        return

    cfg = W.CONFIGS[args.config]
    if args.theta is not None:
        if not 0.0 <= args.theta <= 1.0:
            print("--theta must lie in [0, 1]", file=sys.stderr)
            sys.exit(2)
        cfg = cfg.with_(theta=args.theta)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    B.load_library()
    cfg0 = cfg
    L, (cfg, seg_info, ep_ms, graph_ms, path_fused), ms_step, dom_ms, per_stage_ms, iso_ms, cold_ms, N, counts, \
        stages = \
        time_layer(cfg, args, dev)
    share = parse_share(args.share)

    # algorithmic work per launch
    T, d, E, k, f, s = cfg.T, cfg.d, cfg.E, cfg.top_k, cfg.d_ff, cfg.elem_bytes
    # The library streams the weights through the skinny kernel when the bf16
    # FFN's row capacity (T*k) averages at most 64 rows per segment; that
    # kernel is bound by the weight bytes of the segments that have rows.
    skinny = cfg.dtype == "bf16" and T * k <= 64 * len(counts)
    S_w = sum(1 for c in counts if c > 0)
    work = {
        "route": ("hbm", T * d * s + E * d * s + T * k * 16),
        # fused gather: the permutation only (slot_group in, slot_row and perm_token out)
        "dispatch": ("hbm", (T * k * 8 + N * 4) if path_fused else
                     (T * k * 4 + T * d * s + N * d * s + N * 4 + T * k * 4)),
        "ffn_gate_up": ("hbm", 2 * S_w * d * f * s + N * d * s + N * f * s) if skinny else ("mfma", 4.0 * N * d * f),
        "ffn_down": ("hbm", S_w * d * f * s + N * f * s + N * d * s) if skinny else ("mfma", 2.0 * N * d * f),
        "shared_ffn": ("mfma", 6.0 * T * d * cfg.d_ff_shared),
        "combine": ("hbm", T * k * 8 + N * d * s + T * d * s * (2 if cfg.n_shared else 1)),
    }
    # per stage: "us" and the rates from the stage launched alone back to back,
    # "in_step_us" from events around every stage in a second pass over the
    # same steps (the timed steps carry events only around the dominant kernel)
    stage_out = {}
    for st_name in stages:
        kind, amount = work[st_name]
        ms = iso_ms[st_name]
        if kind == "hbm":
            rate = amount / (ms * 1e-3) / 1e9
            stage_out[st_name] = {"us": round(ms * 1e3, 2), "in_step_us": round(per_stage_ms[st_name] * 1e3, 2),
                                  "bytes": int(amount), "GB_s": round(rate, 1),
                                  "frac_of_hbm_peak": round(rate / HBM_PEAK_GBS, 4)}
            if st_name in cold_ms:
                cold = amount / (cold_ms[st_name] * 1e-3) / 1e9
                stage_out[st_name].update({"cold_us": round(cold_ms[st_name] * 1e3, 2), "cold_GB_s": round(cold, 1),
                                           "cold_frac_of_hbm_peak": round(cold / HBM_PEAK_GBS, 4)})
        else:
            peak = MFMA_BF16_PEAK_TFLOPS if cfg.dtype == "bf16" else VALU_F32_PEAK_TFLOPS
            rate = amount / (ms * 1e-3) / 1e12
            stage_out[st_name] = {"us": round(ms * 1e3, 2), "in_step_us": round(per_stage_ms[st_name] * 1e3, 2),
                                  "flop": amount, "TFLOP_s": round(rate, 1), "frac_of_peak": round(rate / peak, 4)}
            if st_name in cold_ms:
                cold = amount / (cold_ms[st_name] * 1e-3) / 1e12
                stage_out[st_name].update({"cold_us": round(cold_ms[st_name] * 1e3, 2),
                                           "cold_TFLOP_s": round(cold, 1), "cold_frac_of_peak": round(cold / peak, 4)})

    dom = "ffn_gate_up"
    dkind, damount = work[dom]
    dms = dom_ms  # HIP events around the dominant kernel (timed steps, or the per-stage pass)
    # the record holds for the named workload only, not a share or another threshold
    traffic = (recorded_traffic(args.config)
               if share is None and args.theta is None and not path_fused else None)
    if skinny:
        dach = damount / (dms * 1e-3) / 1e9
        cach = damount / (cold_ms[dom] * 1e-3) / 1e9
        kname = "skinny_dma_kernel" if d % 64 == 0 else "skinny_gemm_kernel"
        # the decode weights fit the 256 MB MALL: back-to-back steps read them
        # from there, so the HBM fraction is the cold launch's
        roofline = {"kernel": f"{kname}<gated> (brownout_moe_ffn_gate_up)", "bound": "hbm",
                    "achieved": round(cach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(cach / HBM_PEAK_GBS, 4), "traffic": traffic,
                    "warm_achieved": round(dach, 1), "warm_frac": round(dach / HBM_PEAK_GBS, 4),
                    "per_launch": f"weights 2*S*d*d_ff*s with S={S_w} segments with rows, plus N*d*s rows read and "
                                  f"N*d_ff*s written, N={N}; achieved from cold launches (after a 1 GiB read "
                                  f"pass), warm_* from the timed steps (weights served from the MALL)"}
    else:
        dpeak = MFMA_BF16_PEAK_TFLOPS if cfg.dtype == "bf16" else VALU_F32_PEAK_TFLOPS
        dach = damount / (dms * 1e-3) / 1e12
        roofline = {"kernel": "grouped_gemm_dma_kernel<gated> (brownout_moe_ffn_gate_up)",
                    "bound": "mfma" if cfg.dtype == "bf16" else "alu",
                    "achieved": round(dach, 1), "peak": dpeak, "unit": "TFLOP/s",
                    "frac": round(dach / dpeak, 4), "traffic": traffic,
                    "per_launch": f"4*N*d*d_ff flop, N={N} rows; traffic: HBM bytes per launch (scaled pmc)"}

    result = {
        "metric": "grouped-MoE layer tokens/sec on 1 MI355X; FFN MFMA util %; route/permute HBM GB/s",
        "value": round(cfg.T / (ms_step * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic (seeded numpy PCG64; random-init united-expert weights)",
        "config": {"workload": WORKLOAD_TEXT[args.config], "name": cfg.name, "T": T, "d": d, "E": E,
                   "top_k": k, "G": cfg.G, "d_ff": f, "d_ff_shared": cfg.d_ff_shared,
                   "norm_topk": cfg.norm_topk, "zipf_s": cfg.zipf_s, "seed": args.seed,
                   "rows_N": N, "group_rows": counts},
        "roofline": roofline,
        "stages": stage_out,
        "stages_note": "us / rates: the stage launched alone back to back (warm: activations, and weights "
                       "below 256 MB, may be served from the 256 MB MALL); in_step_us: inside a second pass over the "
                       "steps with events around every stage, one stage after another on one stream; "
                       "cold_*: median launch after a 1 GiB read pass that evicts L2 and the MALL, timed by HIP "
                       "events around the one launch (so it includes the launch and event overhead that "
                       "cold_launch_floor_us measures on a one-workgroup elementwise launch)",
        "cold_launch_floor_us": round(cold_ms["launch_floor"] * 1e3, 2),
        "graph_ms_per_step": None if graph_ms is None else round(graph_ms, 4),
        "graph_note": "one step captured into a HIP graph and replayed `steps` times back to back (wall clock): "
                      "the kernels without the host's per-call launch work; value and ms_per_step are the eager "
                      "steps",
        "cpu_baseline": None,
    }

    # the layer's path: the four calls, or dispatch writing only the
    # permutation and the gate/up GEMM gathering its rows from x (LayerForward
    # takes the latter by default from top-3 on)
    result["config"]["gather"] = "fused" if path_fused else "four calls"
    if seg_info is not None:
        # G above is the united-expert count; the layer ran over the segments
        result["config"]["partial_brownout"] = seg_info
    if share is not None:
        kind, P = share
        if kind == "tp":
            # one rank's share: d_ff above is the share's; the P partial
            # outputs would be summed across the GPUs (not timed here)
            result["config"]["share"] = {"kind": "tensor-parallel", "P": P, "rank": args.share_rank,
                                         "d_ff_full": cfg0.d_ff}
        else:
            offs = np.concatenate([[0], np.cumsum(counts)])
            ranks = []
            for r in range(P):
                g0, g1 = W.ep_groups(cfg.G, P, r)
                ranks.append({"united_experts": [g0, g1], "rows": int(offs[g1] - offs[g0]),
                              "ffn_us": round(ep_ms[r] * 1e3, 2)})
            result["config"]["share"] = {"kind": "expert-parallel", "P": P}
            result["ep_ffn"] = {"ranks": ranks, "straggler_us": max(r["ffn_us"] for r in ranks),
                                "note": "each rank's grouped FFN (gate/up + down) over its block, "
                                        "on the rows the whole dispatch gave it; exchange not timed"}

    if path_fused and not args.fused_gather and not args.no_compare_fused and share is None:
        # the same layer on the four-call path (bit-identical results)
        nargs = argparse.Namespace(**{**vars(args), "four_calls": True})
        _, _, ms_n, _, _, iso_n, _, _, _, _ = time_layer(cfg0, nargs, dev)
        result["four_calls"] = {"value": round(cfg.T / (ms_n * 1e-3), 1), "ms_per_step": round(ms_n, 4),
                                "stages_us": {k: round(v * 1e3, 2) for k, v in iso_n.items()},
                                "fused_speedup": round(ms_n / ms_step, 3),
                                "note": "dispatch writes x_perm and the gate/up GEMM reads it"}
    if not path_fused and not args.no_compare_fused and share is None:
        # the same layer on the fused-gather path (bit-identical results)
        fargs = argparse.Namespace(**{**vars(args), "fused_gather": True})
        _, _, ms_f, _, stages_f, iso_f, _, _, _, _ = time_layer(cfg0, fargs, dev)
        result["fused_gather"] = {"value": round(cfg.T / (ms_f * 1e-3), 1), "ms_per_step": round(ms_f, 4),
                                  "stages_us": {k: round(v * 1e3, 2) for k, v in iso_f.items()},
                                  "speedup": round(ms_step / ms_f, 3),
                                  "note": "dispatch writes only the permutation; the gate/up GEMM gathers "
                                          "its rows from x"}

    if not args.fused_gather and not args.no_compare_fold and share is None and cfg0.dtype == "bf16":
        # the combine folded into the down projection (no stream-K split of its
        # tiles), beside the same layer unfused and without the split
        fargs = argparse.Namespace(**{**vars(args), "fold_combine": True})
        _, _, ms_f, _, _, iso_f, cold_f, _, _, _ = time_layer(cfg0, fargs, dev)
        nargs = argparse.Namespace(**{**vars(args), "no_stream_k": True})
        _, _, ms_n, _, _, iso_n, _, _, _, _ = time_layer(cfg0, nargs, dev)
        result["fold_combine"] = {"value": round(cfg.T / (ms_f * 1e-3), 1), "ms_per_step": round(ms_f, 4),
                                  "stages_us": {k: round(v * 1e3, 2) for k, v in iso_f.items()},
                                  "speedup": round(ms_step / ms_f, 3),
                                  "unsplit_unfused": {"value": round(cfg.T / (ms_n * 1e-3), 1),
                                                      "ms_per_step": round(ms_n, 4),
                                                      "stages_us": {k: round(v * 1e3, 2) for k, v in iso_n.items()}},
                                  "note": "down projection with the combine in its epilogue (tiles never split); "
                                          "unsplit_unfused: the four-call layer without the stream-K workspace, "
                                          "which the fold reproduces bit for bit"}

    plain = share is None and args.theta is None and not args.fused_gather and cfg0.dtype == "bf16"
    if plain and not args.no_compare_ungrouped and cfg0.G != cfg0.E:
        # zero brownout on the same layer: every expert its own group
        result["ungrouped"] = ungrouped_line(cfg0, args, dev, ms_step)

    if plain and args.config == "mixtral" and not args.no_extra:
        # the other full-size workloads, grouped and ungrouped, in the same run
        result["other_workloads"] = {}
        for name in ("fine", "heavy", "decode"):
            wcfg = W.CONFIGS[name]
            xargs = argparse.Namespace(**{**vars(args), "share": None, "fused_gather": False})
            _, (_, _, _, graph_w, fused_w), ms_w, dom_w, _, iso_w, cold_w, N_w, counts_w, _ = \
                time_layer(wcfg, xargs, dev, device_weights=True)
            line = {"workload": WORKLOAD_TEXT[name], "value": round(wcfg.T / (ms_w * 1e-3), 1),
                    "unit": "tokens/s", "ms_per_step": round(ms_w, 4),
                    "gather": "fused" if fused_w else "four calls",
                    "graph_ms_per_step": None if graph_w is None else round(graph_w, 4), "rows_N": N_w,
                    "dominant": dominant_rate(wcfg, N_w, counts_w, dom_w, cold_w["ffn_gate_up"]),
                    "stages_us": {k: round(v * 1e3, 2) for k, v in iso_w.items()},
                    "stages_cold_us": {k: round(v * 1e3, 2) for k, v in cold_w.items()}}
            line["ungrouped"] = ungrouped_line(wcfg, xargs, dev, ms_w)
            result["other_workloads"][name] = line
        result["other_workloads_note"] = ("same kernels and bench protocol; united-expert weights drawn on the "
                                          "device from the workload's distribution (route inputs from the seeded "
                                          "host generator); ungrouped: G = E, every expert its own group (zero "
                                          "brownout), the in-framework analogue of the paper's grouped-vs-unfused "
                                          "comparison (Sec. 5), not comparable with its numbers")

    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(L, cfg0, share, args.share_rank, args.cpu_seconds)

    print(json.dumps(result), flush=True)


def bench_distill(args, dev):
    """One candidate grouping of the search (Sec. 4.3), evaluated on the GPU:
    the united experts start as their members' parameter average, run on the
    T calibration tokens, and the errors of Eq. 5-6 follow. The members'
    outputs are computed once (the calibration run records them) and are not
    part of the timed step."""
    import torch
    from paper_2607_04164_amd import binding as B
    from paper_2607_04164_amd import workload as W

    cfg = W.CONFIGS[args.config]
    if cfg.dtype != "bf16":
        raise SystemExit("--distill runs the bf16 workloads")
    T, d, E, G, f = cfg.T, cfg.d, cfg.E, cfg.G, cfg.d_ff
    print(f"[bench] distill: generating {cfg.name} experts", file=sys.stderr, flush=True)
    L = W.make_layer(cfg, args.seed, with_weights=False)
    parts = [W.expert_weights(L, e) for e in range(E)]
    to_dev = lambda a: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
    we = [to_dev(np.stack([p[j] for p in parts])) for j in range(3)]
    del parts
    x = to_dev(L.x)
    e2g = torch.from_numpy(L.e2g).to(dev)
    wfreq = torch.from_numpy(W.zipf_freq(L).astype(np.float32)).to(dev)
    fws = B.new_ffn_workspace(B.make_desc(T, d, E, cfg.top_k, G, f, 0, 0, "bf16"), dev)
    y_e = B.ffn_all_tokens(x, *we, workspace=fws)  # once per calibration run
    wu = B.united_init(e2g, G, *we)
    offs, a_rows = B.all_tokens_rows(G, T, dev)
    h = torch.empty((G * T, f), dtype=torch.bfloat16, device=dev)
    y_u = torch.empty((G * T, d), dtype=torch.bfloat16, device=dev)
    dws = torch.empty(B.DISTILL_WS_BYTES, dtype=torch.uint8, device=dev)
    mse = torch.zeros(G, dtype=torch.float64, device=dev)
    tot = torch.zeros((), dtype=torch.float64, device=dev)
    stages = {
        "united_init": lambda: B.united_init(e2g, G, *we, out=wu),
        "united_ffn": lambda: B.ffn_gather(offs, a_rows, x, *wu, h=h, y=y_u, workspace=fws),
        "distill_mse": lambda: B.distill_mse(e2g, wfreq, y_e, y_u, T, workspace=dws, out=(mse, tot)),
    }

    def step():
        for fn in stages.values():
            fn()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / args.steps
    s = 2
    work = {"united_init": ("hbm", 3 * (E + G) * d * f * s), "united_ffn": ("mfma", 6.0 * G * T * d * f),
            "distill_mse": ("hbm", (E + G) * T * d * s)}
    out = {}
    for name, fn in stages.items():
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        reps = 3 if name == "united_ffn" else 10
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        sms = e0.elapsed_time(e1) / reps
        kind, amt = work[name]
        if kind == "hbm":
            rate = amt / (sms * 1e-3) / 1e9
            out[name] = {"us": round(sms * 1e3, 2), "bytes": int(amt), "GB_s": round(rate, 1),
                         "frac_of_hbm_peak": round(rate / HBM_PEAK_GBS, 4)}
        else:
            rate = amt / (sms * 1e-3) / 1e12
            out[name] = {"us": round(sms * 1e3, 2), "flop": amt, "TFLOP_s": round(rate, 1),
                         "frac_of_peak": round(rate / MFMA_BF16_PEAK_TFLOPS, 4)}
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    B.ffn_all_tokens(x, *we, workspace=fws)
    e1.record()
    torch.cuda.synchronize()
    mse_h = mse.cpu().numpy().tolist()
    dom = out["united_ffn"]
    result = {
        "metric": "grouping candidates evaluated per second (united init + united-expert FFN on the "
                  "calibration tokens + routing-weighted distillation errors), 1 MI355X",
        "value": round(1e3 / ms, 2), "unit": "candidates/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic (seeded expert weights and tokens)",
        "config": {"workload": f"grouping search on the {cfg.name} layer: E={E} experts, G={G} united, d={d}, "
                               f"d_ff={f}, T={T} calibration tokens, zero distillation steps",
                   "E": E, "G": G, "d": d, "d_ff": f, "T": T},
        "roofline": {"kernel": "grouped_gemm_dma_kernel<gated> + <down> (united-expert FFN, gathered rows)",
                     "bound": "mfma", "achieved": dom["TFLOP_s"], "peak": MFMA_BF16_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": dom["frac_of_peak"], "traffic": None},
        "stages": out,
        "expert_outputs_once_us": round(e0.elapsed_time(e1) * 1e3, 1),
        "mse": [round(v, 6) for v in mse_h], "mse_total": round(float(tot.item()), 6),
    }
    print(json.dumps(result), flush=True)


def host_cpu():
    """The host's CPU model, logical CPUs and the CPUs this process may use."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except AttributeError:
        usable = os.cpu_count()
    return {"cpu_model": model, "nproc": os.cpu_count(), "usable_cpus": usable}


def oracle_layer_timed(Lf):
    """The oracle's whole layer (the same stage calls as oracle.layer), each
    stage timed; returns (seconds per stage, total seconds)."""
    import oracle
    cfg = Lf.cfg
    st = {}
    t = time.perf_counter()
    x = Lf.x
    r = oracle.route(x, Lf.w_router, Lf.bias, Lf.e2g, cfg.top_k, cfg.norm_topk)
    st["route"] = time.perf_counter() - t
    t = time.perf_counter()
    dsp = oracle.dispatch(r["slot_group"], cfg.G)
    xp = oracle.gather_rows(x, dsp["perm_token"])
    st["dispatch"] = time.perf_counter() - t
    t = time.perf_counter()
    y = oracle.ffn(dsp["offsets"], xp, Lf.w_gate, Lf.w_up, Lf.w_down)
    st["ffn"] = time.perf_counter() - t
    y_sh = None
    if cfg.n_shared:
        t = time.perf_counter()
        y_sh = oracle.ffn(np.array([0, cfg.T], np.int32), x, Lf.w_gate_sh, Lf.w_up_sh, Lf.w_down_sh)
        st["shared_ffn"] = time.perf_counter() - t
    t = time.perf_counter()
    oracle.combine(dsp["slot_row"], r["slot_gate"], y, y_sh, d=cfg.d)
    st["combine"] = time.perf_counter() - t
    return st, sum(st.values())


def widen(L):
    """The layer with its bf16 storage widened to the float32 the oracle reads."""
    import dataclasses
    names = ("x", "w_router", "w_gate", "w_up", "w_down", "w_gate_sh", "w_up_sh", "w_down_sh")
    return dataclasses.replace(L, cfg=L.cfg.with_(dtype="f32"), **{k: L.f32(k) for k in names})


def cpu_baseline(L, cfg, share, rank, budget_s):
    """The CPU oracle, unchanged, on a bounded sample of the same tokens (of
    the same share of the layer when it is sharded), stage by stage; and, for
    reference, the whole tiny and decode workloads on one thread and on all."""
    import dataclasses

    import oracle
    from oracle.partial import partial_map
    from paper_2607_04164_amd import workload as W

    if cfg.theta is not None:
        # the oracle's own segment map for partial brownout
        e2s, seg = partial_map(W.zipf_freq(L), L.e2g, cfg.G, cfg.theta)
        L = W.segment_layer(L, e2s, seg)
        cfg = L.cfg
    if share and share[0] == "tp":
        L = W.tp_share(L, share[1], rank)
        cfg = L.cfg

    # widen the bf16 storage to the float32 the oracle reads, once, outside the timing
    Lf = widen(L)

    def run(n):
        sub = dataclasses.replace(Lf, cfg=Lf.cfg.with_(T=n), x=Lf.x[:n])
        return oracle_layer_timed(sub)

    print("[bench] cpu baseline (oracle)", file=sys.stderr, flush=True)
    run(min(4, cfg.T))  # warm caches once
    n0 = min(16, cfg.T)
    st, t0 = run(n0)
    n = int(min(cfg.T, max(n0, n0 * budget_s / max(t0, 1e-6))))
    if n != n0:
        st, t = run(n)
    else:
        t = t0
    threads = oracle.num_threads()
    out = {"value": round(n / t, 2), "unit": "tokens/s", "cores": threads, "kind": "oracle",
           "sample": f"first {n} of {cfg.T} tokens of the same workload, whole layer "
                     f"(route, dispatch, FFN, combine), {t:.1f} s wall on {threads} threads",
           "stages_s": {k: round(v, 4) for k, v in st.items()}}
    out.update(host_cpu())
    # whole small workloads, one thread and all threads
    single = {}
    for name in ("tiny", "decode"):
        Ls = widen(W.make_layer(W.CONFIGS[name], 0))
        row = {}
        for nt in (1, threads):
            oracle.set_num_threads(nt)
            oracle_layer_timed(Ls)  # warm
            best = min(oracle_layer_timed(Ls)[1] for _ in range(3))
            row[f"tokens_s_{nt}_threads"] = round(Ls.cfg.T / best, 2)
        oracle.set_num_threads(threads)
        single[name] = row
    out["whole_small_workloads"] = single
    return out


if __name__ == "__main__":
    main()
