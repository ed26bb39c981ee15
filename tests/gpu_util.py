"""Helpers shared by the GPU parity tests: moving seeded workloads to the
device, calling the oracle on the same bytes, and the comparison rules.

Comparison rules (the bar each parity test applies):
  * integer and index outputs (top-k indices, group ids, counts, offsets,
    permutation, slot rows) and copied rows (x_perm): bit-exact;
  * gate weights (topk_w, slot_gate): relative error <= 1e-5 (fp32 softmax
    against the oracle's float64 one, rounded once);
  * bf16 FFN outputs (h, y_perm) and the layer output: the largest absolute
    error in a row, divided by that row's largest |oracle value|, <= 1e-2
    (inputs exact in bf16, fp32 accumulation, three bf16 roundings of about
    2^-9 relative each on the way: h, y and out);
  * fp32 configurations: the same row-max-relative error <= 1e-4.
"""
from __future__ import annotations

import numpy as np
import torch

import oracle
from paper_2607_04164_amd import binding as B
from paper_2607_04164_amd import workload as W

TOL = {"bf16": 1e-2, "f32": 1e-4}
GATE_RTOL = 1e-5


def desc_of(cfg: W.LayerConfig) -> B.Desc:
    return B.make_desc(cfg.T, cfg.d, cfg.E, cfg.top_k, cfg.G, cfg.d_ff, cfg.d_ff_shared,
                       cfg.norm_topk, cfg.dtype)


def dev_tensor(a: np.ndarray, dtype: str, device="cuda") -> torch.Tensor:
    """Storage-format numpy array (float32, or uint16 bf16 bits) -> device tensor."""
    if dtype == "bf16" and a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


def host_f32(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy()


def to_storage(a_f32: np.ndarray, dtype: str) -> np.ndarray:
    return W.f32_to_bf16_bits(a_f32) if dtype == "bf16" else np.ascontiguousarray(a_f32, np.float32)


def device_weights(L: W.Layer, device="cuda"):
    dt = L.cfg.dtype
    w = {
        "w_router": dev_tensor(L.w_router, dt, device),
        "bias": torch.from_numpy(L.bias).to(device),
        "e2g": torch.from_numpy(L.e2g.astype(np.int32)).to(device),
        "w_gate": dev_tensor(L.w_gate, dt, device),
        "w_up": dev_tensor(L.w_up, dt, device),
        "w_down": dev_tensor(L.w_down, dt, device),
    }
    if L.cfg.n_shared:
        w["w_gate_sh"] = dev_tensor(L.w_gate_sh, dt, device)
        w["w_up_sh"] = dev_tensor(L.w_up_sh, dt, device)
        w["w_down_sh"] = dev_tensor(L.w_down_sh, dt, device)
    return w


def rowmax_rel_err(got, ref) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    if got.size == 0:
        return 0.0
    den = np.maximum(np.abs(ref).max(axis=-1, keepdims=True), 1e-30)
    return float((np.abs(got - ref) / den).max())


def assert_close_rows(got, ref, dtype: str, what: str):
    err = rowmax_rel_err(got, ref)
    assert np.all(np.isfinite(got)), f"{what}: non-finite values"
    assert err <= TOL[dtype], f"{what}: row-max relative error {err:.3e} > {TOL[dtype]}"
    return err


def assert_gates(got, ref, what: str):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    err = np.abs(got - ref) / np.maximum(np.abs(ref), 1e-30)
    err[(ref == 0) & (got == 0)] = 0.0
    assert float(err.max(initial=0.0)) <= GATE_RTOL, f"{what}: relative error {err.max():.3e}"


def group_boundary_tokens(perm_token: np.ndarray, offsets: np.ndarray) -> np.ndarray:
    """Tokens that own the first and last row of every non-empty group segment."""
    out = []
    for r in range(len(offsets) - 1):
        if offsets[r + 1] > offsets[r]:
            out += [perm_token[offsets[r]], perm_token[offsets[r + 1] - 1]]
    return np.unique(np.array(out, dtype=np.int64))


def stream_k_split_rows(offsets, n_cols, K, gated: bool, n_cu: int, split_min_idle: int = 48):
    """Rows of every output tile whose K loop the persistent 256-row GEMM
    splits across workgroups (stream-K) when it runs with the FFN workspace.

    This restates the kernel's tile schedule only to choose which rows a
    parity test samples (a mistake here weakens the sample, it cannot make a
    wrong result pass): segments in order, inside a segment groups of 8
    M-tiles of 256 rows with the N-tiles outer; P = the CU count rounded down
    to a multiple of 8 workgroups; whole rounds of one tile per workgroup,
    and the K-steps (64 columns each) of the tiles after them split evenly
    when whole tiles would leave the workgroups idle for more than
    split_min_idle K-steps on average (only the last partial round when that
    gives every workgroup at least 8 K-steps, else the last one to two)."""
    BM, BN, BK, GM = 256, (128 if gated else 256), 64, 8
    P = n_cu // 8 * 8
    offs = [int(o) for o in offsets]
    n_seg = len(offs) - 1
    mts = [-(-(offs[s + 1] - offs[s]) // BM) for s in range(n_seg)]
    NT = -(-n_cols // BN)
    total = sum(mts) * NT
    nk = K // BK
    if P == 0 or total == 0 or K % BK:
        return np.zeros(0, np.int64)
    rounds = -(-total // P)
    if (rounds * P - total) * nk <= split_min_idle * P:
        return np.zeros(0, np.int64)
    full = total // P
    rest = (total - full * P) * nk
    F = full if rest >= 8 * P else max(0, full - 1)
    first_mt = np.concatenate([[0], np.cumsum(mts)])
    rows = set()
    for L in range(F * P, total):
        s = int(np.searchsorted(first_mt * NT, L, side="right") - 1)
        local = L - first_mt[s] * NT
        mg = local // (GM * NT)
        gm = min(GM, mts[s] - mg * GM)
        mt = mg * GM + (local - mg * GM * NT) % gm
        r0 = offs[s] + mt * BM
        rows.update(range(r0, min(r0 + BM, offs[s + 1])))
    return np.array(sorted(rows), np.int64)
