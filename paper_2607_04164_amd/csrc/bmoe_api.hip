// Host side of the C ABI: argument checks (host only, before anything is
// enqueued), workspace sizing, status strings and the four entry points.
#include <limits.h>

#include "bmoe_common.h"

namespace {

using namespace bmoe;

inline bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

inline int elem_bytes(int dtype) { return dtype == BMOE_BF16 ? 2 : 4; }

inline bmoe_status hip_status(hipError_t e) { return e == hipSuccess ? BMOE_OK : BMOE_ERR_HIP; }

}  // namespace

extern "C" {

int32_t bmoe_version(void) { return 10000; }

const char* bmoe_status_str(bmoe_status s) {
    switch (s) {
        case BMOE_OK: return "ok";
        case BMOE_ERR_NULL: return "a required pointer is NULL";
        case BMOE_ERR_SHAPE: return "a size is out of range";
        case BMOE_ERR_ALIGN: return "a tensor pointer is not 16-byte aligned";
        case BMOE_ERR_MAP: return "an expert-to-group map entry is outside [0, G)";
        case BMOE_ERR_UNSUPPORTED: return "unsupported dtype or mode";
        case BMOE_ERR_WORKSPACE: return "workspace missing or too small";
        case BMOE_ERR_HIP: return "HIP runtime error at launch";
    }
    return "unknown status";
}

bmoe_status bmoe_validate(const bmoe_desc* d) {
    if (!d) return BMOE_ERR_NULL;
    if (d->dtype != BMOE_F32 && d->dtype != BMOE_BF16) return BMOE_ERR_UNSUPPORTED;
    if (d->T < 0 || d->E < 1 || d->E > BMOE_MAX_EXPERTS) return BMOE_ERR_SHAPE;
    if (d->top_k < 1 || d->top_k > d->E || d->top_k > BMOE_MAX_TOPK) return BMOE_ERR_SHAPE;
    if (d->G < 1 || d->G > d->E) return BMOE_ERR_SHAPE;
    if (d->d < 8 || d->d % 8 != 0 || d->d_ff < 8 || d->d_ff % 8 != 0) return BMOE_ERR_SHAPE;
    if (d->d_ff_shared < 0 || d->d_ff_shared % 8 != 0) return BMOE_ERR_SHAPE;
    if (d->norm_topk != 0 && d->norm_topk != 1) return BMOE_ERR_SHAPE;
    // row indices (T*k) and element offsets within a row fit 32-bit ints
    if ((int64_t)d->T * d->top_k > INT_MAX / 2) return BMOE_ERR_SHAPE;
    if (d->d > (1 << 20) || d->d_ff > (1 << 20) || d->d_ff_shared > (1 << 20)) return BMOE_ERR_SHAPE;
    return BMOE_OK;
}

bmoe_status bmoe_validate_map(const int32_t* e2g, int32_t E, int32_t G) {
    if (!e2g) return BMOE_ERR_NULL;
    if (E < 1 || E > BMOE_MAX_EXPERTS || G < 1 || G > E) return BMOE_ERR_SHAPE;
    for (int e = 0; e < E; ++e)
        if (e2g[e] < 0 || e2g[e] >= G) return BMOE_ERR_MAP;
    return BMOE_OK;
}

size_t bmoe_workspace_bytes(const bmoe_desc* d, int32_t stage) {
    if (bmoe_validate(d) != BMOE_OK) return 0;
    if (stage == BMOE_STAGE_DISPATCH) return dispatch_ws_bytes(d->T, d->G);
    if (stage == BMOE_STAGE_FFN && d->dtype == BMOE_BF16) return ffn_workspace_bytes();
    if (stage == BMOE_STAGE_DOWN_COMBINE) return down_combine_ws_bytes(d->T, d->d);
    return 0;
}

bmoe_status brownout_moe_route(const bmoe_desc* d, const void* x, const void* w_router,
                               const float* bias, const float* logits_in, const int32_t* e2g,
                               int32_t* topk_idx, float* topk_w, int32_t* slot_group, float* slot_gate,
                               float* logits_out, void* stream) {
    bmoe_status st = bmoe_validate(d);
    if (st != BMOE_OK) return st;
    if (d->T == 0) return BMOE_OK;
    if (!e2g || !topk_idx || !topk_w || !slot_group || !slot_gate) return BMOE_ERR_NULL;
    if (!logits_in && (!x || !w_router)) return BMOE_ERR_NULL;
    if (!logits_in && (!aligned16(x) || !aligned16(w_router))) return BMOE_ERR_ALIGN;
    RouteArgs a{x, w_router, bias, logits_in, e2g, topk_idx, topk_w, slot_group, slot_gate, logits_out,
                d->T, d->d, d->E, d->top_k, d->G, d->norm_topk, d->dtype};
    return hip_status(launch_route(a, (hipStream_t)stream));
}

bmoe_status brownout_moe_dispatch(const bmoe_desc* d, const int32_t* slot_group, const void* x,
                                  int32_t* counts, int32_t* offsets, int32_t* perm_token,
                                  int32_t* slot_row, void* x_perm, void* ws, size_t ws_bytes,
                                  void* stream) {
    bmoe_status st = bmoe_validate(d);
    if (st != BMOE_OK) return st;
    if (d->T == 0) return BMOE_OK;
    // x_perm NULL: the permutation only (x is then not read and may be NULL)
    if (!slot_group || !counts || !offsets || !perm_token || !slot_row || (x_perm && !x))
        return BMOE_ERR_NULL;
    if (x_perm && (!aligned16(x) || !aligned16(x_perm))) return BMOE_ERR_ALIGN;
    if (!ws || ws_bytes < dispatch_ws_bytes(d->T, d->G)) return BMOE_ERR_WORKSPACE;
    if (((uintptr_t)ws & 255u) != 0) return BMOE_ERR_ALIGN;
    DispatchArgs a{slot_group, x, counts, offsets, perm_token, slot_row, x_perm, ws,
                   d->T, d->d, d->top_k, d->G, elem_bytes(d->dtype)};
    return hip_status(launch_dispatch(a, (hipStream_t)stream));
}

bmoe_status brownout_moe_dispatch_noalloc(const bmoe_desc* d, const int32_t* slot_group, const void* x,
                                          int32_t* counts, int32_t* offsets, int32_t* perm_token,
                                          int32_t* slot_row, void* x_perm, void* stream) {
    bmoe_status st = bmoe_validate(d);
    if (st != BMOE_OK) return st;
    if (d->T == 0) return BMOE_OK;
    if (!slot_group || !counts || !offsets || !perm_token || !slot_row || (x_perm && !x))
        return BMOE_ERR_NULL;
    if (x_perm && (!aligned16(x) || !aligned16(x_perm))) return BMOE_ERR_ALIGN;
    if (dispatch_ws_bytes(d->T, d->G) > (size_t)BMOE_DISPATCH_SCRATCH_BYTES) return BMOE_ERR_WORKSPACE;
    DispatchArgs a{slot_group, x, counts, offsets, perm_token, slot_row, x_perm, nullptr,
                   d->T, d->d, d->top_k, d->G, elem_bytes(d->dtype)};
    return hip_status(launch_dispatch_noalloc(a, (hipStream_t)stream));
}

}  // extern "C"

namespace {

// a_rows != nullptr: the gate/up GEMM reads row r of its A operand from
// a[a_rows[r]], a holding a_count rows
bmoe_status ffn_common(int part, int32_t dtype, int32_t n_seg, int32_t rows_cap, int32_t d, int32_t d_ff,
                       const int32_t* offsets, const void* a, const void* w_gate, const void* w_up,
                       const void* w_down, void* h, void* y, void* ws, size_t ws_bytes, void* stream,
                       const int32_t* a_rows = nullptr, int32_t a_count = 0, int32_t split_min_idle = -1) {
    if (dtype != BMOE_F32 && dtype != BMOE_BF16) return BMOE_ERR_UNSUPPORTED;
    if (n_seg < 1 || n_seg > BMOE_MAX_EXPERTS || rows_cap < 0) return BMOE_ERR_SHAPE;
    if (d < 8 || d % 8 != 0 || d_ff < 8 || d_ff % 8 != 0) return BMOE_ERR_SHAPE;
    if (d > (1 << 20) || d_ff > (1 << 20)) return BMOE_ERR_SHAPE;
    if ((int64_t)rows_cap * (d > d_ff ? d : d_ff) > ((int64_t)1 << 40)) return BMOE_ERR_SHAPE;
    if (rows_cap == 0) return BMOE_OK;
    const bool up = part != 2, down = part != 1;
    if (!offsets || !h) return BMOE_ERR_NULL;
    if (up && (!a || !w_gate || !w_up)) return BMOE_ERR_NULL;
    if (down && (!w_down || !y)) return BMOE_ERR_NULL;
    if (!aligned16(h)) return BMOE_ERR_ALIGN;
    if (up && (!aligned16(a) || !aligned16(w_gate) || !aligned16(w_up))) return BMOE_ERR_ALIGN;
    if (down && (!aligned16(w_down) || !aligned16(y))) return BMOE_ERR_ALIGN;
    if (ws && ((uintptr_t)ws & 255u)) return BMOE_ERR_ALIGN;
    if (dtype != BMOE_BF16) ws = nullptr;  // the fp32 kernels take no workspace
    if (ws && ws_bytes < ffn_workspace_bytes()) return BMOE_ERR_WORKSPACE;
    if (split_min_idle < -1 || split_min_idle > (1 << 20)) return BMOE_ERR_SHAPE;
    FfnArgs args{offsets, a, w_gate, w_up, w_down, h, y, ws, ws_bytes, n_seg, rows_cap, d, d_ff, dtype};
    args.split_min_idle = split_min_idle;
    if (a_rows) {
        // the copy kernels address a gathered source with 32-bit byte offsets
        if (a_count < 1 || (int64_t)a_count * d * elem_bytes(dtype) >= ((int64_t)1 << 32)) return BMOE_ERR_SHAPE;
        args.a_rows = a_rows;
        args.a_count = a_count;
    }
    return hip_status(launch_ffn(args, (hipStream_t)stream, part));
}

}  // namespace

extern "C" {

bmoe_status brownout_moe_ffn(int32_t dtype, int32_t n_seg, int32_t rows_cap, int32_t d, int32_t d_ff,
                             const int32_t* offsets, const void* a, const void* w_gate,
                             const void* w_up, const void* w_down, void* h, void* y, void* workspace,
                             size_t workspace_bytes, void* stream) {
    return ffn_common(0, dtype, n_seg, rows_cap, d, d_ff, offsets, a, w_gate, w_up, w_down, h, y, workspace,
                      workspace_bytes, stream);
}

bmoe_status brownout_moe_ffn_ex(int32_t dtype, int32_t n_seg, int32_t rows_cap, int32_t d, int32_t d_ff,
                                const int32_t* offsets, const void* a, const void* w_gate, const void* w_up,
                                const void* w_down, void* h, void* y, void* workspace, size_t workspace_bytes,
                                int32_t split_min_idle, void* stream) {
    return ffn_common(0, dtype, n_seg, rows_cap, d, d_ff, offsets, a, w_gate, w_up, w_down, h, y, workspace,
                      workspace_bytes, stream, nullptr, 0, split_min_idle);
}

bmoe_status brownout_moe_ffn_gather(int32_t dtype, int32_t n_seg, int32_t rows_cap, int32_t d, int32_t d_ff,
                                    const int32_t* offsets, const int32_t* a_rows, int32_t a_count,
                                    const void* a, const void* w_gate, const void* w_up, const void* w_down,
                                    void* h, void* y, void* workspace, size_t workspace_bytes, void* stream) {
    if (rows_cap > 0 && !a_rows) return BMOE_ERR_NULL;
    return ffn_common(0, dtype, n_seg, rows_cap, d, d_ff, offsets, a, w_gate, w_up, w_down, h, y, workspace,
                      workspace_bytes, stream, a_rows, a_count);
}

bmoe_status brownout_moe_ffn_gate_up_gather(int32_t dtype, int32_t n_seg, int32_t rows_cap, int32_t d,
                                            int32_t d_ff, const int32_t* offsets, const int32_t* a_rows,
                                            int32_t a_count, const void* a, const void* w_gate, const void* w_up,
                                            void* h, void* workspace, size_t workspace_bytes, void* stream) {
    if (rows_cap > 0 && !a_rows) return BMOE_ERR_NULL;
    return ffn_common(1, dtype, n_seg, rows_cap, d, d_ff, offsets, a, w_gate, w_up, nullptr, h, nullptr,
                      workspace, workspace_bytes, stream, a_rows, a_count);
}

bmoe_status brownout_moe_ffn_gate_up(int32_t dtype, int32_t n_seg, int32_t rows_cap, int32_t d,
                                     int32_t d_ff, const int32_t* offsets, const void* a,
                                     const void* w_gate, const void* w_up, void* h, void* workspace,
                                     size_t workspace_bytes, void* stream) {
    return ffn_common(1, dtype, n_seg, rows_cap, d, d_ff, offsets, a, w_gate, w_up, nullptr, h, nullptr,
                      workspace, workspace_bytes, stream);
}

bmoe_status brownout_moe_ffn_down(int32_t dtype, int32_t n_seg, int32_t rows_cap, int32_t d, int32_t d_ff,
                                  const int32_t* offsets, const void* h, const void* w_down, void* y,
                                  void* workspace, size_t workspace_bytes, void* stream) {
    // h is only read by the down GEMM
    return ffn_common(2, dtype, n_seg, rows_cap, d, d_ff, offsets, nullptr, nullptr, nullptr, w_down,
                      const_cast<void*>(h), y, workspace, workspace_bytes, stream);
}

bmoe_status brownout_moe_ffn_down_combine(const bmoe_desc* d, const int32_t* offsets, const void* h,
                                          const void* w_down, void* y, const int32_t* perm_token,
                                          const int32_t* slot_row, const float* slot_gate, const void* y_shared,
                                          void* out, void* workspace, size_t workspace_bytes, void* stream) {
    bmoe_status st = bmoe_validate(d);
    if (st != BMOE_OK) return st;
    if (d->T == 0) return BMOE_OK;
    if (!offsets || !h || !w_down || !y || !perm_token || !slot_row || !slot_gate || !out) return BMOE_ERR_NULL;
    if (!aligned16(h) || !aligned16(w_down) || !aligned16(y) || !aligned16(out) ||
        (y_shared && !aligned16(y_shared)))
        return BMOE_ERR_ALIGN;
    const int32_t rows_cap = d->T * d->top_k;
    if ((int64_t)rows_cap * (d->d > d->d_ff ? d->d : d->d_ff) > ((int64_t)1 << 40)) return BMOE_ERR_SHAPE;
    if (!workspace || workspace_bytes < down_combine_ws_bytes(d->T, d->d)) return BMOE_ERR_WORKSPACE;
    if ((uintptr_t)workspace & 255u) return BMOE_ERR_ALIGN;
    FfnArgs args{offsets, nullptr, nullptr, nullptr, w_down, const_cast<void*>(h), y, nullptr, 0,
                 d->G, rows_cap, d->d, d->d_ff, d->dtype};
    args.fold.perm_token = perm_token;
    args.fold.slot_row = slot_row;
    args.fold.slot_gate = slot_gate;
    args.fold.y_shared = (const uint16_t*)y_shared;
    args.fold.out = (uint16_t*)out;
    args.fold.cnt = (int32_t*)workspace;
    args.fold.k = d->top_k;
    if (ffn_can_fold(args)) return hip_status(launch_ffn(args, (hipStream_t)stream, 2));
    // other shapes: the down projection, then the combine kernel
    args.fold = FoldArgs{};
    hipError_t e = launch_ffn(args, (hipStream_t)stream, 2);
    if (e != hipSuccess) return BMOE_ERR_HIP;
    CombineArgs c{slot_row, slot_gate, y, y_shared, out, d->T, d->top_k, d->d, elem_bytes(d->dtype),
                  (int64_t)rows_cap};
    return hip_status(launch_combine(c, (hipStream_t)stream));
}

bmoe_status brownout_moe_united_init(int32_t dtype, int32_t E, int32_t G, int32_t d, int32_t d_ff,
                                     const int32_t* e2g, const void* w_gate_e, const void* w_up_e,
                                     const void* w_down_e, void* w_gate_u, void* w_up_u, void* w_down_u,
                                     void* stream) {
    if (dtype != BMOE_F32 && dtype != BMOE_BF16) return BMOE_ERR_UNSUPPORTED;
    if (E < 1 || E > BMOE_MAX_EXPERTS || G < 1 || G > BMOE_MAX_EXPERTS) return BMOE_ERR_SHAPE;
    if (d < 8 || d % 8 != 0 || d_ff < 8 || d_ff % 8 != 0 || d > (1 << 20) || d_ff > (1 << 20))
        return BMOE_ERR_SHAPE;
    if (!e2g || !w_gate_e || !w_up_e || !w_down_e || !w_gate_u || !w_up_u || !w_down_u) return BMOE_ERR_NULL;
    for (const void* p : {w_gate_e, w_up_e, w_down_e, (const void*)w_gate_u, (const void*)w_up_u,
                          (const void*)w_down_u})
        if (!aligned16(p)) return BMOE_ERR_ALIGN;
    bmoe::UnitedInitArgs a{e2g, {w_gate_e, w_up_e, w_down_e}, {w_gate_u, w_up_u, w_down_u}, E, G, d, d_ff, dtype};
    return hip_status(bmoe::launch_united_init(a, (hipStream_t)stream));
}

bmoe_status brownout_moe_distill_mse(int32_t dtype, int32_t E, int32_t G, int32_t T, int32_t d,
                                     const int32_t* e2g, const float* w_freq, const void* y_expert,
                                     const void* y_united, double* mse, double* mse_total, void* workspace,
                                     size_t workspace_bytes, void* stream) {
    if (dtype != BMOE_F32 && dtype != BMOE_BF16) return BMOE_ERR_UNSUPPORTED;
    if (E < 1 || E > BMOE_MAX_EXPERTS || G < 1 || G > BMOE_MAX_EXPERTS || T < 0) return BMOE_ERR_SHAPE;
    if (d < 8 || d % 8 != 0 || d > (1 << 20)) return BMOE_ERR_SHAPE;
    if (T == 0) return BMOE_OK;
    const int nb = bmoe::distill_blocks(G, T);
    // the partial kernel indexes a workgroup's chunks with 32-bit ints
    if ((int64_t)((T + nb - 1) / nb + 1) * (d / (dtype == BMOE_BF16 ? 8 : 4)) >= ((int64_t)1 << 31))
        return BMOE_ERR_SHAPE;
    if (!e2g || !w_freq || !y_expert || !y_united || !mse) return BMOE_ERR_NULL;
    if (!aligned16(y_expert) || !aligned16(y_united) || ((uintptr_t)mse & 7u) || ((uintptr_t)mse_total & 7u))
        return BMOE_ERR_ALIGN;
    if (!workspace || workspace_bytes < (size_t)nb * G * sizeof(double)) return BMOE_ERR_WORKSPACE;
    if ((uintptr_t)workspace & 7u) return BMOE_ERR_ALIGN;
    bmoe::DistillArgs a{e2g, w_freq, y_expert, y_united, mse, mse_total, workspace, E, G, T, d, dtype};
    return hip_status(bmoe::launch_distill_mse(a, (hipStream_t)stream));
}

bmoe_status brownout_moe_combine(const bmoe_desc* d, const int32_t* slot_row, const float* slot_gate,
                                 const void* y_perm, const void* y_shared, void* out, void* stream) {
    bmoe_status st = bmoe_validate(d);
    if (st != BMOE_OK) return st;
    if (d->T == 0) return BMOE_OK;
    if (!slot_row || !slot_gate || !y_perm || !out) return BMOE_ERR_NULL;
    if (!aligned16(y_perm) || !aligned16(out) || (y_shared && !aligned16(y_shared))) return BMOE_ERR_ALIGN;
    CombineArgs a{slot_row, slot_gate, y_perm, y_shared, out, d->T, d->top_k, d->d, elem_bytes(d->dtype),
                  (int64_t)d->T * d->top_k};
    return hip_status(launch_combine(a, (hipStream_t)stream));
}

}  // extern "C"
