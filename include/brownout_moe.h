/*
 * brownout_moe.h -- C ABI of the grouped ("full-brownout") MoE layer forward
 * for AMD Instinct MI355X (gfx950).
 *
 * The layer (paper: Sec. 2.1 for the top-K MoE layer, Eq. 1-2 in Sec. 4.2 for
 * the expert-to-group map, the closing paragraphs of Sec. 4.3 and Sec. 4.4 for
 * how the map is used while serving): a gate picks each token's top-k experts
 * among E; a map g sends expert e to united expert g(e) of G; under full
 * brownout every picked expert is served by its united expert. A token whose
 * picks share a united expert calls it once with the sum of their gate
 * weights. The output is
 *
 *     out_t = sum over distinct groups r of t's picks of gamma_{t,r} * FFN_r(x_t)
 *             (+ shared-expert FFN(x_t) when the layer has shared experts)
 *
 * with FFN_r a SwiGLU expert, y = W_down (silu(W_gate a) * (W_up a)).
 *
 * Four calls make one forward, enqueued on one stream with no host sync:
 *   brownout_moe_route     gate logits, softmax, top-k, map, per-group merge
 *   brownout_moe_dispatch  per-group histogram, prefix, stable permutation, row gather
 *   brownout_moe_ffn       grouped SwiGLU FFN over the united experts
 *   brownout_moe_combine   gate-weighted sum back into token order
 *
 * Conventions for every call:
 *   - Tensor pointers are DEVICE pointers, row-major, owned by the caller. The
 *     library allocates and frees nothing at run time. Its only device memory
 *     is two fixed arrays of its code object, one copy per GPU: 64 KiB of
 *     zeros that the FFN's copies of padding rows read, and the workspace of
 *     brownout_moe_dispatch_noalloc. On the host it caches per-device facts
 *     (CU count, those arrays' addresses, kernel attributes set once).
 *   - Weights use the [out, in] layout: W_gate/W_up [n, d_ff, d], W_down [n, d, d_ff].
 *   - Every call checks its arguments on the host before it enqueues anything;
 *     on error it returns a BMOE_ERR_* code and writes nothing. Launch failures
 *     return BMOE_ERR_HIP. Calls are asynchronous on `stream` (a hipStream_t;
 *     NULL is the default stream); outputs are valid once the stream has
 *     reached them.
 *   - Pointers to float/bf16 tensors that kernels read or write 16 bytes at a
 *     time (x, x_perm, w_*, h, y, out, y_shared) must be 16-byte aligned; d and
 *     d_ff must be multiples of 8.
 *   - T == 0 is a no-op that returns BMOE_OK.
 *   - Inputs must be finite.
 */
#ifndef BROWNOUT_MOE_H
#define BROWNOUT_MOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__)
#define BMOE_API __attribute__((visibility("default")))
#else
#define BMOE_API
#endif

#define BMOE_MAX_EXPERTS 256 /* E <= 256, hence G <= 256 */
#define BMOE_MAX_TOPK 16     /* top_k <= 16 */

/* Route decides every token whose fast fp32 logits leave any two of its top
 * (k+1) values closer than this gap (2^-14) again from float64 logits; see
 * brownout_moe_route. The gap is far above the error of the fp32 logits (a few
 * 1e-6 at d = 4096), so every pair the fp32 logits order is ordered the same
 * way by the float64 ones. */
#define BMOE_ROUTE_RECHECK_GAP (1.0f / 16384.0f)

typedef enum bmoe_status {
    BMOE_OK = 0,
    BMOE_ERR_NULL = 1,        /* a required pointer is NULL                       */
    BMOE_ERR_SHAPE = 2,       /* a size is out of range                            */
    BMOE_ERR_ALIGN = 3,       /* a pointer is not 16-byte aligned                  */
    BMOE_ERR_MAP = 4,         /* an expert-to-group map entry is outside [0, G)    */
    BMOE_ERR_UNSUPPORTED = 5, /* unknown dtype, or a mode this build does not do  */
    BMOE_ERR_WORKSPACE = 6,   /* workspace missing or too small                    */
    BMOE_ERR_HIP = 7          /* the HIP runtime reported an error at launch       */
} bmoe_status;

typedef enum bmoe_dtype {
    BMOE_F32 = 0,  /* float activations and weights                        */
    BMOE_BF16 = 1  /* bf16 activations and weights, fp32 accumulation      */
} bmoe_dtype;

typedef enum bmoe_stage {
    BMOE_STAGE_ROUTE = 0,
    BMOE_STAGE_DISPATCH = 1,
    BMOE_STAGE_FFN = 2,
    BMOE_STAGE_COMBINE = 3,
    BMOE_STAGE_DOWN_COMBINE = 4  /* brownout_moe_ffn_down_combine */
} bmoe_stage;

/* Shape of one layer. */
typedef struct bmoe_desc {
    int32_t T;           /* tokens, >= 0                                          */
    int32_t d;           /* model width, multiple of 8                            */
    int32_t E;           /* routed experts, 1..256                                */
    int32_t top_k;       /* experts per token, 1..min(E, 16)                      */
    int32_t G;           /* united experts (groups), 1..E                         */
    int32_t d_ff;        /* SwiGLU width of a united expert, multiple of 8        */
    int32_t d_ff_shared; /* width of the always-on shared FFN, 0 = none           */
    int32_t norm_topk;   /* 1: the k gate weights are renormalised to sum to 1    */
    int32_t dtype;       /* bmoe_dtype                                            */
} bmoe_desc;

/* Host-only checks (no HIP call). */
BMOE_API bmoe_status bmoe_validate(const bmoe_desc* desc);
/* e2g_host[E] (host memory): every entry in [0, G). The map is a static
 * per-layer artifact (Sec. 4.3-4.4); kernels assume a validated map. */
BMOE_API bmoe_status bmoe_validate_map(const int32_t* e2g_host, int32_t E, int32_t G);
/* Workspace bytes a stage needs for `desc` (0: none). */
BMOE_API size_t bmoe_workspace_bytes(const bmoe_desc* desc, int32_t stage);
/* Static string for a status code. */
BMOE_API const char* bmoe_status_str(bmoe_status status);
/* Library version, e.g. 10000 for 1.0.0. */
BMOE_API int32_t bmoe_version(void);

/*
 * bmoe_partial_segment_map -- host only: the segment map of partial brownout.
 * Paper: Sec. 2.2 (zero, partial and full brownout), Sec. 5 baselines
 * (threshold 1.0 keeps every original expert, 0 substitutes every call),
 * Sec. 4.3 closing paragraph (only eligible cold calls are replaced through
 * the saved map), Sec. 4.5 (the controller moves the threshold).
 *
 * Hot experts: the longest run of experts in order of decreasing freq (ties:
 * lower index first) whose cumulative freq / sum(freq) is <= theta + 1e-9.
 * Segments: the hot experts in ascending index (each with its own FFN), then
 * the united experts with at least one cold member in ascending group index.
 * The layer runs over the segments with e2s in place of e2g and S = *n_seg
 * in place of G (the weights of segment s stacked at index s).
 *
 * freq[E] double (calibration routing frequencies: finite, >= 0, positive
 * sum), e2g[E] int32 in [0, G), theta in [0, 1]; all HOST memory. Outputs,
 * host memory: e2s[E] int32; seg_kind[E] int32 (0: a hot expert's own FFN,
 * 1: a united expert) and seg_id[E] int32 (that expert or group), first
 * *n_seg entries valid; *n_seg in 1..E. Errors: BMOE_ERR_NULL,
 * BMOE_ERR_SHAPE (sizes, theta, frequencies), BMOE_ERR_MAP (e2g); nothing
 * is written on error.
 */
BMOE_API bmoe_status bmoe_partial_segment_map(const double* freq, const int32_t* e2g, int32_t E, int32_t G,
                                             double theta, int32_t* e2s, int32_t* seg_kind, int32_t* seg_id,
                                             int32_t* n_seg);

/*
 * brownout_moe_route -- the gate and the substitution by united experts.
 * Paper: Sec. 2.1 (gating scores g_i of the top-K experts), Eq. 2 (the map),
 * Sec. 4.3 last paragraph before Algorithm 1 (the gate still picks the
 * experts; picked experts are replaced by their united expert).
 *
 *   z[t,e]   = x[t,:] . w_router[e,:] + bias[e]          (or logits_in[t,e])
 *   p[t,:]   = softmax over all E of z[t,:]
 *   slot i   = the i-th largest z[t,:] (ties: lower expert index first)
 *   topk_idx[t,i] = that expert; topk_w[t,i] = its p (divided by the sum of
 *                   the k values when desc->norm_topk)
 *   slot_group[t,i] = e2g[topk_idx[t,i]] if no earlier slot of t has that
 *                   group, else -1;
 *   slot_gate[t,i]  = sum of topk_w[t,j] over j >= i with the same group when
 *                   slot_group[t,i] >= 0, else 0.
 *
 * x [T,d] (dtype), w_router [E,d] (dtype), bias [E] float or NULL, e2g [E]
 * int32 (validated map), logits_in [T,E] float or NULL. When logits_in is
 * set, x, w_router and bias are not used (they may be NULL) and selection
 * runs on those exact values.
 * Otherwise the logits are computed in fp32 (bf16: MFMA); a token whose fp32
 * top-(k+1) values have an adjacent gap below BMOE_ROUTE_RECHECK_GAP has its
 * candidate experts re-evaluated in float64 and is selected on those.
 * Outputs: topk_idx, slot_group [T,k] int32; topk_w, slot_gate [T,k] float;
 * logits_out [T,E] float or NULL (the fp32 logits, bias included).
 * No workspace.
 */
BMOE_API bmoe_status brownout_moe_route(const bmoe_desc* desc, const void* x, const void* w_router,
                               const float* bias, const float* logits_in, const int32_t* e2g,
                               int32_t* topk_idx, float* topk_w, int32_t* slot_group,
                               float* slot_gate, float* logits_out, void* stream);

/*
 * brownout_moe_dispatch -- group rows for the united experts (Eq. 2: the sets
 * G_r of the map, here filled with (token, group) pairs).
 *
 *   counts[r]   = number of tokens with a valid slot of group r
 *   offsets     = exclusive prefix of counts, offsets[G] = N (total rows)
 *   rows of group r are offsets[r] .. offsets[r+1]-1, in ascending token order
 *   perm_token[row] = token of that row; slot_row[t,i] = row of slot (t,i), or -1
 *   x_perm[row,:]   = x[perm_token[row],:]  (bit copy)
 *
 * slot_group [T,k] int32 as written by brownout_moe_route (entries outside
 * [-1, G) count as -1). x [T,d] (dtype). counts [G], offsets [G+1],
 * perm_token [T*k], slot_row [T,k] int32; x_perm [T*k, d] (dtype). Rows at
 * and beyond N are left unspecified.
 * x_perm NULL: the permutation only (counts, offsets, perm_token, slot_row);
 * no row is copied and x is not read (it may be NULL). This is the first half
 * of the fused path, whose FFN gathers its rows from x through perm_token
 * (brownout_moe_ffn_gather).
 * workspace: bmoe_workspace_bytes(desc, BMOE_STAGE_DISPATCH) bytes, 256-byte
 * aligned, ALL ZERO before the first call that uses it; every call leaves it
 * all zero again when it completes on the stream. Two calls that share a
 * workspace must not overlap in time. A call that finds the workspace not
 * zero (for example after an earlier call on it was cut short) writes the
 * "no rows" result instead: counts all 0, offsets[0..G-1] = 0 and
 * offsets[G] = -1 (the sentinel to check), every slot_row -1, no row copied;
 * the FFN and combine then see no rows. It still leaves the workspace zero.
 * Implementation: a histogram with LDS atomics and a single-pass decoupled
 * look-back scan across token tiles, then a 128-bit row gather; at most 256
 * tokens (one tile) take one kernel in which every workgroup rebuilds the
 * tile's histogram and prefix in LDS before gathering its tokens' rows.
 */
BMOE_API bmoe_status brownout_moe_dispatch(const bmoe_desc* desc, const int32_t* slot_group,
                                  const void* x, int32_t* counts, int32_t* offsets,
                                  int32_t* perm_token, int32_t* slot_row, void* x_perm,
                                  void* workspace, size_t workspace_bytes, void* stream);

/*
 * brownout_moe_dispatch_noalloc -- brownout_moe_dispatch for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation): the same kernels and results, but
 * the workspace is a device array inside the library, one per GPU, of
 * BMOE_DISPATCH_SCRATCH_BYTES bytes, held until the process ends. The call
 * allocates nothing; each call first clears the array with a kernel (no
 * memset, so it may be captured into a graph). Arguments as for
 * brownout_moe_dispatch without the workspace. Shapes whose workspace
 * (bmoe_workspace_bytes(desc, BMOE_STAGE_DISPATCH)) exceeds the array return
 * BMOE_ERR_WORKSPACE before anything is enqueued. Every call on one GPU uses
 * that GPU's array, which keeps the last call's contents: two calls on one GPU
 * that overlap in time (other streams, other threads) race and must not be
 * made. The device is the current HIP device.
 */
#define BMOE_DISPATCH_SCRATCH_BYTES 1048576
BMOE_API bmoe_status brownout_moe_dispatch_noalloc(const bmoe_desc* desc, const int32_t* slot_group,
                                          const void* x, int32_t* counts, int32_t* offsets,
                                          int32_t* perm_token, int32_t* slot_row, void* x_perm,
                                          void* stream);

/*
 * brownout_moe_ffn -- grouped SwiGLU FFN (Sec. 2.1 "small FFNs"; SwiGLU form).
 * Segment s covers rows offsets[s] .. offsets[s+1]-1 of a and uses united
 * expert s:
 *   h[row,:] = silu(a[row,:] W_gate[s]^T) * (a[row,:] W_up[s]^T)   (stored in dtype)
 *   y[row,:] = h[row,:] W_down[s]^T                                  (stored in dtype)
 * dtype: bmoe_dtype. offsets [n_seg+1] int32 in DEVICE memory (as written by
 * dispatch; non-decreasing, offsets[n_seg] <= rows_cap; rows beyond rows_cap
 * are never touched). a [rows_cap, d]; w_gate, w_up [n_seg, d_ff, d];
 * w_down [n_seg, d, d_ff]; h [rows_cap, d_ff] (scratch the caller owns);
 * y [rows_cap, d]. n_seg in 1..256. bf16: MFMA, fp32 accumulation.
 * offsets[0] need not be 0: a sub-range of segments runs alone when the
 * caller passes offsets + s0 and the weights of segments s0.. (one rank's
 * block of united experts under expert parallelism); other rows stay untouched.
 * The shared experts of a layer run through this call too, with n_seg = 1,
 * offsets = {0, T}, a = x.
 * workspace (optional, device memory, 256-byte aligned): the large bf16
 * GEMMs run one workgroup per CU, each taking whole output tiles in turn;
 * NULL keeps every tile whole. With at least bmoe_workspace_bytes(desc,
 * BMOE_STAGE_FFN) bytes (the size depends on the current device) they may
 * also split the K loop of the last tiles so every CU gets the same work;
 * the partial sums of a split tile meet in the workspace in a fixed order,
 * so results stay deterministic (they may differ in the last bits from the
 * NULL-workspace path). Contents need no
 * initialisation and are not preserved; calls that can overlap in time must
 * not share a workspace. A non-NULL workspace below the size is
 * BMOE_ERR_WORKSPACE. The K loops are split only when whole tiles would leave
 * the CUs idle for more than 48 K-steps (of 64 columns) on average
 * (brownout_moe_ffn_ex takes that threshold as an argument).
 */
BMOE_API bmoe_status brownout_moe_ffn(int32_t dtype, int32_t n_seg, int32_t rows_cap, int32_t d,
                             int32_t d_ff, const int32_t* offsets, const void* a,
                             const void* w_gate, const void* w_up, const void* w_down, void* h,
                             void* y, void* workspace, size_t workspace_bytes, void* stream);

/* brownout_moe_ffn with the stream-K split threshold given explicitly: with a
 * workspace, the K loops of the last tiles are split when whole tiles would
 * leave the CUs idle for more than split_min_idle K-steps (of 64 columns) on
 * average; 0 splits whenever any CU would idle, -1 takes the default (48).
 * Values below -1 or above 2^20 are BMOE_ERR_SHAPE. The result is the same
 * layer as brownout_moe_ffn's within the rounding of the split sums. */
BMOE_API bmoe_status brownout_moe_ffn_ex(int32_t dtype, int32_t n_seg, int32_t rows_cap, int32_t d,
                                int32_t d_ff, const int32_t* offsets, const void* a,
                                const void* w_gate, const void* w_up, const void* w_down, void* h,
                                void* y, void* workspace, size_t workspace_bytes,
                                int32_t split_min_idle, void* stream);

/* The two grouped GEMMs of brownout_moe_ffn, callable on their own (same
 * arguments and rules as brownout_moe_ffn):
 *   brownout_moe_ffn_gate_up: h = silu(a W_gate[s]^T) * (a W_up[s]^T)
 *   brownout_moe_ffn_down:    y = h W_down[s]^T                                   */
BMOE_API bmoe_status brownout_moe_ffn_gate_up(int32_t dtype, int32_t n_seg, int32_t rows_cap, int32_t d,
                                     int32_t d_ff, const int32_t* offsets, const void* a,
                                     const void* w_gate, const void* w_up, void* h, void* workspace,
                                     size_t workspace_bytes, void* stream);
BMOE_API bmoe_status brownout_moe_ffn_down(int32_t dtype, int32_t n_seg, int32_t rows_cap, int32_t d,
                                  int32_t d_ff, const int32_t* offsets, const void* h,
                                  const void* w_down, void* y, void* workspace, size_t workspace_bytes,
                                  void* stream);

/* Fused gather (the same FFN, Sec. 2.1, without the x_perm copy): the gate/up
 * GEMM reads row r of its activations as a[a_rows[r], :] instead of a[r, :],
 * straight from the token rows: with a = x [T, d], a_count = T and a_rows =
 * the perm_token that brownout_moe_dispatch wrote (with x_perm NULL there),
 * the results are bit-identical to dispatch's x_perm followed by
 * brownout_moe_ffn. a_rows [rows_cap] int32 in DEVICE memory; entries are
 * clamped into [0, a_count) (never read out of bounds); a [a_count, d]
 * (dtype), 16-byte aligned; a_count * d * element size must stay below
 * 2^32 bytes (BMOE_ERR_SHAPE otherwise). NULL a_rows with rows_cap > 0 is
 * BMOE_ERR_NULL. Every other argument and rule as brownout_moe_ffn /
 * brownout_moe_ffn_gate_up; the down GEMM is unchanged (h is already in row
 * order). */
BMOE_API bmoe_status brownout_moe_ffn_gather(int32_t dtype, int32_t n_seg, int32_t rows_cap, int32_t d,
                                    int32_t d_ff, const int32_t* offsets, const int32_t* a_rows,
                                    int32_t a_count, const void* a, const void* w_gate, const void* w_up,
                                    const void* w_down, void* h, void* y, void* workspace,
                                    size_t workspace_bytes, void* stream);
BMOE_API bmoe_status brownout_moe_ffn_gate_up_gather(int32_t dtype, int32_t n_seg, int32_t rows_cap, int32_t d,
                                            int32_t d_ff, const int32_t* offsets, const int32_t* a_rows,
                                            int32_t a_count, const void* a, const void* w_gate,
                                            const void* w_up, void* h, void* workspace,
                                            size_t workspace_bytes, void* stream);

/*
 * Grouping search (Sec. 4.3): what a candidate map costs in distillation
 * error. The member experts' outputs f_e(x) and the united experts' outputs
 * f_u(x) on the calibration tokens come from brownout_moe_ffn_gather with one
 * segment per expert (rows e*T .. e*T+T-1 read token t = row mod T).
 *
 * brownout_moe_united_init -- the united experts' starting point: each united
 * matrix is the element-wise average of its members' matrices (the parameter
 * average the paper starts distillation from, Sec. 4.3, after Eq. 5).
 *   w_*_u[r] = (sum over e with e2g[e] == r, ascending e, of w_*_e[e]) / count
 * e2g [E] int32 in DEVICE memory (entries outside [0, G) belong to no group);
 * w_gate_e, w_up_e [E, d_ff, d], w_down_e [E, d, d_ff]; w_gate_u, w_up_u
 * [G, d_ff, d], w_down_u [G, d, d_ff] (dtype; bf16: fp32 sum, rounded once;
 * f32: fp64 sum). An empty group gets zeros. E, G in 1..256.
 */
BMOE_API bmoe_status brownout_moe_united_init(int32_t dtype, int32_t E, int32_t G, int32_t d, int32_t d_ff,
                                     const int32_t* e2g, const void* w_gate_e, const void* w_up_e,
                                     const void* w_down_e, void* w_gate_u, void* w_up_u, void* w_down_u,
                                     void* stream);

/*
 * brownout_moe_distill_mse -- distillation error of every group and the
 * layer total (Eq. 5, Eq. 3 and Eq. 6):
 *   alpha_e  = w_e / (sum of w over e's group)  (equal weights if that sum is 0)
 *   t_r(x_t) = sum over the members e of r of alpha_e y_expert[e*T + t, :]
 *   mse[r]   = mean over t < T and j < d of (y_united[r*T + t, j] - t_r(x_t)[j])^2
 *   *mse_total = sum over r of beta_r mse[r],  beta_r = sum of w over r's members
 * (the reward of the grouping search is -*mse_total). An empty group has
 * mse 0 and beta 0. e2g [E] int32 and w_freq [E] float (routing frequencies)
 * in DEVICE memory; y_expert [E*T, d], y_united [G*T, d] (dtype, 16-byte
 * aligned); mse [G] double, mse_total (nullable) double, in DEVICE memory.
 * Targets in fp32, squares accumulated in fp64 in a fixed order: results are
 * deterministic. workspace: at least BMOE_DISTILL_WS_BYTES bytes of device
 * memory, 8-byte aligned, contents need no initialisation (calls that can
 * overlap must not share one). T == 0 writes nothing.
 */
#define BMOE_DISTILL_WS_BYTES 32768
BMOE_API bmoe_status brownout_moe_distill_mse(int32_t dtype, int32_t E, int32_t G, int32_t T, int32_t d,
                                     const int32_t* e2g, const float* w_freq, const void* y_expert,
                                     const void* y_united, double* mse, double* mse_total, void* workspace,
                                     size_t workspace_bytes, void* stream);

/*
 * brownout_moe_ffn_down_combine -- the down projection with the combine folded
 * into its epilogue (the fused MoE operator of Sec. 4.1; the layer output of
 * Sec. 2.1). Writes the same y as brownout_moe_ffn_down and the same out, bit
 * for bit, as brownout_moe_combine on that y (fp32 fmaf of slot gate and bf16
 * y over the token's valid slots in slot order, + y_shared, one RNE rounding),
 * whatever order the tiles finish in: each tile's epilogue counts its rows per
 * (token, 128-column chunk), and the row that completes a token's chunk forms
 * that chunk of out from the token's rows of y.
 * desc: the layer (G segments, d, d_ff, top_k, dtype). offsets [G+1], h
 * [T*k, d_ff], w_down [G, d, d_ff], y [T*k, d], perm_token [T*k], slot_row
 * [T,k], slot_gate [T,k] (as written by route and dispatch), y_shared [T,d] or
 * NULL, out [T,d]. workspace: bmoe_workspace_bytes(desc,
 * BMOE_STAGE_DOWN_COMBINE) bytes (4 * T * ceil(d/128)), 256-byte aligned, ALL
 * ZERO before the first call; every call leaves it zero; calls that share one
 * must not overlap. The fold runs on the 256-row bf16 GEMM tiles with d a
 * multiple of 128 (every tile whole: no stream-K split); other shapes run the
 * down projection and then the combine kernel, with the same results.
 */
BMOE_API bmoe_status brownout_moe_ffn_down_combine(const bmoe_desc* desc, const int32_t* offsets, const void* h,
                                          const void* w_down, void* y, const int32_t* perm_token,
                                          const int32_t* slot_row, const float* slot_gate,
                                          const void* y_shared, void* out, void* workspace,
                                          size_t workspace_bytes, void* stream);

/*
 * brownout_moe_combine -- weighted sum back into token order (Sec. 2.1: the
 * layer output is the gate-weighted sum of the expert outputs).
 *   out[t,:] = sum over i ascending with slot_row[t,i] >= 0 of
 *              slot_gate[t,i] * y_perm[slot_row[t,i],:]  (+ y_shared[t,:])
 * fp32 accumulation, stored in dtype. slot_row [T,k] int32, slot_gate [T,k]
 * float, y_perm [T*k, d], y_shared [T,d] or NULL, out [T,d]. Rows of y_perm
 * named by slot_row must be < T*k.
 */
BMOE_API bmoe_status brownout_moe_combine(const bmoe_desc* desc, const int32_t* slot_row,
                                 const float* slot_gate, const void* y_perm,
                                 const void* y_shared, void* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* BROWNOUT_MOE_H */
