// Gate and united-expert substitution (paper Sec. 2.1 gating, Eq. 2 map,
// Sec. 4.3 closing paragraph: the gate picks experts, the map replaces them).
//
// One workgroup (4 waves) owns BT = 16*TB tokens:
//   1. logits tile [BT, E] into LDS:
//        bf16: x rows and W_router rows are copied straight into LDS
//              (global_load_lds, swizzled rows) in super-chunks of KS*KW*64
//              columns through a ring of slots shared by the 4 waves;
//              16x16x32 bf16 MFMA, fp32 accumulate; with KS > 1 the waves
//              split the d axis and their partial tiles are summed in LDS
//              in a fixed order;
//        bf16, E <= 8, d a multiple of 1024 up to 4096: 16 tokens, the
//              waves split d; each wave loads its x columns straight into
//              registers (all at once) and copies its W_router columns into
//              its own LDS area, so the copy phase has no barrier;
//        f32:  one (token, expert) dot product per thread;
//        logits_in: copied.
//   2. per token, a group of S lanes (S <= 16, chosen so that a wave's tokens
//      fill it) holds the E logits, V <= 16 per lane; k+1 rounds of a
//      branch-free local scan and a group arg-max (DPP within rows of 16
//      lanes) give the picks in order (ties: lower expert index); the arg-max
//      key packs the expert id with its united expert, so a round touches no
//      memory. If two adjacent values among the top k+1 are closer than
//      BMOE_ROUTE_RECHECK_GAP the token is queued for step 3. Otherwise
//      softmax, optional renormalisation and the per-group merge are done
//      from the token's pick list and written out.
//   3. queued tokens are decided again in float64 by teams of waves (a lone
//      token gets all four, each summing a quarter of the row): every expert
//      whose fp32 logit is within the gap of the k-th value is recomputed
//      from exact float64 products, and the top-k is taken among those by
//      ranking them.
#include "bmoe_common.h"

#include <atomic>

namespace bmoe {
namespace {

constexpr int kRouteThreads = 256;
constexpr float kGap = BMOE_ROUTE_RECHECK_GAP;
constexpr int kMaxK = BMOE_MAX_TOPK;
static_assert(BMOE_MAX_EXPERTS <= kRouteThreads, "one map entry per thread");

// MODE_BF16: x and W_router through the LDS ring; MODE_BF16_RES: x straight
// into registers, each wave's columns of W_router in its own LDS area (E <= 8,
// d = 1024 * NBAT, NBAT <= 4)
// MODE_BF16_XD: 32 tokens, 17..64 experts, d = 64 * NU (NU in 8, 16, 32): x
// straight into registers, W_router alone through an LDS ring
enum { MODE_LOGITS_IN = 0, MODE_F32 = 1, MODE_BF16 = 2, MODE_BF16_RES = 3, MODE_BF16_XD = 4 };
__host__ __device__ constexpr bool mode_bf16(int mode) { return mode >= MODE_BF16; }

// KW of MODE_BF16_XD carries NU (k-steps of 32 columns per wave, low 6 bits)
// and NS (ring slots, the bits above)
__host__ __device__ constexpr int xd_nu(int kw) { return kw & 63; }
__host__ __device__ constexpr int xd_ns(int kw) { return kw >> 6; }
constexpr int kXdSlot = 16 * 1024;        // 64 router rows x 2 column halves x 64 columns, bf16
constexpr int kXdPart = 2 * 16 * 64 * 4;  // partial tiles of the waves of the second half

// LDS of the router columns (8 rows of d, four wave areas) and of the
// partial logit tiles of waves 1..3
__host__ __device__ inline size_t res_w_bytes(int d) { return (size_t)8 * d * 2; }
constexpr size_t kResPartBytes = 3 * 16 * 16 * 4;

struct RouteSmem {
    int zstride;
    size_t zs_bytes, flag_bytes, cand_bytes, dummy_bytes, ring_bytes;
    __host__ __device__ size_t total() const { return zs_bytes + flag_bytes + cand_bytes + dummy_bytes + ring_bytes; }
};

template <int TB, int NBLK, int KW>
struct RouteCfg {
    // KW: 64-column units each wave multiplies per super-chunk
    static constexpr int BT = 16 * TB, KS = 4 / TB, KC = 64 * KS * KW, EP = 16 * NBLK;
    static constexpr int CPR = KC / 8;                // 16-byte chunks per LDS row
    static constexpr int RPD = 64 / CPR;              // rows per DMA instruction (1 KB)
    static constexpr int SWZ = CPR >= 16 ? 15 : 7;    // swizzle mask of the chunk index
    static constexpr int ROWB = KC * 2;
    static constexpr int XDMA = BT / RPD, WDMA = EP / RPD, TOT = XDMA + WDMA;
    static constexpr int DPW = (TOT + 3) / 4;         // DMA instructions per wave per slot
    static constexpr int SLOT = (BT + EP) * ROWB;
    static constexpr int ZS = (BT * (EP + 1) * 4 + 15) / 16 * 16;
    static constexpr int FLAG = 2048;              // queue of near-tie tokens + map
    static constexpr int DUMMY = 4 * 1024;            // 1 KB per wave for padding copies
    static constexpr int CAND = 4 * 2048;             // per-wave picks / candidate lists
    static constexpr int NSLOT_FIT = (160 * 1024 - ZS - FLAG - CAND - DUMMY) / SLOT;
    static constexpr int NSLOT = NSLOT_FIT > 8 ? 8 : NSLOT_FIT;
    static constexpr int PART = (KS - 1) * BT * EP * 4;
    static constexpr int TOTAL = ZS + FLAG + CAND + DUMMY + NSLOT * SLOT;
    static_assert(NSLOT >= 2, "at least two slots");
    static_assert(CPR <= 64, "a copy instruction covers whole rows");
    static_assert(PART <= NSLOT * SLOT, "partials alias the ring");
    static_assert(TOTAL <= 160 * 1024, "LDS of one workgroup");
    static_assert(DPW * (NSLOT - 2) <= 63, "vmcnt range");
};

template <int MODE, int TB, int NBLK, int KW>
__host__ __device__ inline RouteSmem route_smem(int E, int d) {
    RouteSmem s;
    const int bt = 16 * TB;
    const int e_pad = mode_bf16(MODE) ? 16 * NBLK : ((E + 15) / 16) * 16;
    s.zstride = e_pad + 1;
    s.zs_bytes = ((size_t)bt * s.zstride * 4 + 15) / 16 * 16;
    s.flag_bytes = 2048;
    s.cand_bytes = 4 * 2048;
    s.dummy_bytes = (MODE == MODE_BF16 || MODE == MODE_BF16_XD) ? 4 * 1024 : 0;
    s.ring_bytes = 0;
    if constexpr (MODE == MODE_BF16) s.ring_bytes = (size_t)RouteCfg<TB, NBLK, KW>::NSLOT * RouteCfg<TB, NBLK, KW>::SLOT;
    if constexpr (MODE == MODE_BF16_RES) s.ring_bytes = res_w_bytes(d) + kResPartBytes;
    if constexpr (MODE == MODE_BF16_XD) s.ring_bytes = (size_t)xd_ns(KW) * kXdSlot + kXdPart;
    return s;
}

__device__ __forceinline__ bool better(float v, int e, float bv, int be) {
    return v > bv || (v == bv && e < be);
}
__device__ __forceinline__ bool better(double v, int e, double bv, int be) {
    return v > bv || (v == bv && e < be);
}

// ---- lane exchanges. Within rows of 16 lanes, DPP row permutations (quad
// xor 1, quad xor 2, half-row mirror, row mirror) run on the VALU; they pair
// every lane with a lane of the other half of its group at each step, so
// after log2(S) steps all S lanes of an aligned group hold the reduction.
// Steps across rows (16, 32) go through ds_bpermute (__shfl_xor).
template <int CTRL>
__device__ __forceinline__ int dpp_i(int v) {
    return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
    return __int_as_float(dpp_i<CTRL>(__float_as_int(v)));
}
template <int CTRL>
__device__ __forceinline__ double dpp_d(double v) {
    return __hiloint2double(dpp_i<CTRL>(__double2hiint(v)), dpp_i<CTRL>(__double2loint(v)));
}
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppHalfMirror = 0x141, kDppMirror = 0x140;

template <int CTRL, typename V>
__device__ __forceinline__ void argmax_step(V& bv, int& be) {
    V ov;
    if constexpr (sizeof(V) == 8) ov = dpp_d<CTRL>(bv);
    else ov = dpp_f<CTRL>(bv);
    const int oe = dpp_i<CTRL>(be);
    if (better(ov, oe, bv, be)) { bv = ov; be = oe; }
}

// arg-max (ties: lower index) over aligned groups of S lanes, S in {1,2,4,...,64}
template <int S, typename V>
__device__ __forceinline__ void group_argmax(V& bv, int& be) {
    if constexpr (S >= 2) argmax_step<kDppXor1>(bv, be);
    if constexpr (S >= 4) argmax_step<kDppXor2>(bv, be);
    if constexpr (S >= 8) argmax_step<kDppHalfMirror>(bv, be);
    if constexpr (S >= 16) argmax_step<kDppMirror>(bv, be);
#pragma unroll
    for (int off = 16; off < S; off <<= 1) {
        V ov = __shfl_xor(bv, off);
        int oe = __shfl_xor(be, off);
        if (better(ov, oe, bv, be)) { bv = ov; be = oe; }
    }
}

// sum over aligned groups of S lanes (every lane gets the same bits: each
// step adds two values in an order-independent way)
template <int S, typename V>
__device__ __forceinline__ V group_sum(V v) {
    if constexpr (sizeof(V) == 8) {
        if constexpr (S >= 2) v += dpp_d<kDppXor1>(v);
        if constexpr (S >= 4) v += dpp_d<kDppXor2>(v);
        if constexpr (S >= 8) v += dpp_d<kDppHalfMirror>(v);
        if constexpr (S >= 16) v += dpp_d<kDppMirror>(v);
    } else {
        if constexpr (S >= 2) v += dpp_f<kDppXor1>(v);
        if constexpr (S >= 4) v += dpp_f<kDppXor2>(v);
        if constexpr (S >= 8) v += dpp_f<kDppHalfMirror>(v);
        if constexpr (S >= 16) v += dpp_f<kDppMirror>(v);
    }
#pragma unroll
    for (int off = 16; off < S; off <<= 1) v += __shfl_xor(v, off);
    return v;
}

// A pick in a token's pick list: expert id in the high bits, united expert + 1
// in the low 16 bits (0: the map sends the expert nowhere, so the slot calls
// none). Keys of distinct experts order like their expert ids, so the packed
// value serves as the tie-break index of an arg-max.
constexpr int kNoPick = 0x7fff0000;  // out-of-range expert, no united expert
__device__ __forceinline__ int pack_pick(int e, const int* e2g_s, int E) {
    const int g = (unsigned)e < (unsigned)E ? e2g_s[e] : -1;  // NaN logits pick nothing
    return ((e & 0x7fff) << 16) | (g + 1);
}
__device__ __forceinline__ int pick_expert(int pk) { return pk >> 16; }
__device__ __forceinline__ int pick_group(int pk) { return (pk & 0xffff) - 1; }

// Softmax weights, optional renormalisation and per-group merge of one token
// from its pick list (pk: packed picks, pkv: their logits, largest first),
// shared by the S lanes of the token's group; lane s writes slots s, s+S, ...
// (at most 4 of them: S >= 4 or S >= k). The weight of a pick is
// exp(v - top) / sum_exp, or exp(v - top) / sum over the k picks when the top-k
// weights are renormalised. Exponents are taken in fp32 of the difference,
// far below the gate tolerance.
template <typename V>
__device__ __forceinline__ void finish_token(const RouteArgs& p, int t, int s, int S, const int* pk, const V* pkv,
                                             V top, float sum_exp, bool write) {
    const int k = p.k;
    int gq[4];
    float eq[4], gs[4];
    bool dup[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int q = s + i * S;
        gq[i] = q < k ? pick_group(pk[q]) : -3;
        eq[i] = 0.f;
        gs[i] = 0.f;
        dup[i] = false;
    }
    float tot = 0.f;
#pragma unroll 4
    for (int j = 0; j < k; ++j) {
        const int g = pick_group(pk[j]);
        const float ex = __expf((float)(pkv[j] - top));
        tot += ex;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int q = s + i * S;
            if (j == q) eq[i] = ex;
            if (g == gq[i]) {
                if (j < q) dup[i] = true;
                else gs[i] += ex;
            }
        }
    }
    if (!write) return;
    const float inv = 1.f / (p.norm ? tot : sum_exp);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int q = s + i * S;
        if (q >= k) break;
        const size_t o = (size_t)t * k + q;
        p.topk_idx[o] = pick_expert(pk[q]);
        p.topk_w[o] = eq[i] * inv;
        const bool valid = !dup[i] && gq[i] >= 0;
        p.slot_group[o] = valid ? gq[i] : -1;
        p.slot_gate[o] = valid ? gs[i] * inv : 0.f;
    }
}

// The same from picks held in registers (k <= kRegK; every lane of the
// token's group holds all of them): no memory round trips and no branches
// but the stores. Sums are taken in the same order as above, so the results
// are the same bits.
constexpr int kRegK = 8;
template <typename V>
__device__ __forceinline__ void finish_regs(const RouteArgs& p, int t, int s, int S, const int (&hk)[kRegK],
                                            const V (&hv)[kRegK], float sum_exp, bool write) {
    const int k = p.k;
    float ex[kRegK];
    int g[kRegK];
    float tot = 0.f;
#pragma unroll
    for (int j = 0; j < kRegK; ++j) {
        const bool in = j < k;
        ex[j] = in ? __expf((float)(hv[j] - hv[0])) : 0.f;
        g[j] = in ? pick_group(hk[j]) : -2 - j;  // never equal to a pick's group
        tot += ex[j];
    }
    if (!write) return;
    const float inv = 1.f / (p.norm ? tot : sum_exp);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int q = s + i * S;
        int kq = kNoPick, gq = -2 - kRegK;
        float eq = 0.f;
#pragma unroll
        for (int j = 0; j < kRegK; ++j) {
            kq = j == q ? hk[j] : kq;
            gq = j == q ? g[j] : gq;
            eq = j == q ? ex[j] : eq;
        }
        float gs = 0.f;
        bool dup = false;
#pragma unroll
        for (int j = 0; j < kRegK; ++j) {
            const bool same = g[j] == gq;
            dup = dup || (same && j < q);
            gs += (same && j >= q) ? ex[j] : 0.f;
        }
        if (q < k) {
            const size_t o = (size_t)t * k + q;
            p.topk_idx[o] = pick_expert(kq);
            p.topk_w[o] = eq * inv;
            const bool valid = !dup && gq >= 0;
            p.slot_group[o] = valid ? gq : -1;
            p.slot_gate[o] = valid ? gs * inv : 0.f;
        }
    }
}

// Step 2 for the TPW tokens of one wave. Groups of S lanes are independent
// (their exchanges stay inside the group), so a group without a token idles.
struct SelectCtx {
    const float* zs;
    int zstride;
    int* area;        // the wave's pick area: 32 words per token
    const int* e2g_s;
    int* fl_count;    // the wave's queue of near-tie tokens
    int* fl_tok;
    float* fl_thr;
    int t0, tw0;      // first token of the workgroup, first local row of the wave
    bool recheck;
};

template <int S, int V, int TPW>
__device__ __forceinline__ void select_tokens(const RouteArgs& p, const SelectCtx& c, int lane) {
    constexpr int P = kWave / S;
    const int E = p.E, k = p.k;
    const int s = lane % S, seg = lane / S;
    const int R = min(k + 1, E);
    // this lane holds experts s, s+S, ... below E (vpl <= V of them); the other
    // value slots start out taken, so the rounds need no bounds test
    const int vpl = (E - s + S - 1) / S;
    const unsigned dead = vpl >= V ? 0u : ~0u << vpl;
    int key[V];
#pragma unroll
    for (int j = 0; j < V; ++j) {
        const int e = s + j * S;
        key[j] = j < vpl ? pack_pick(e, c.e2g_s, E) : kNoPick;
    }
#pragma unroll
    for (int base = 0; base < TPW; base += P) {
        const int tw = base + seg;
        if (tw >= TPW) continue;
        const bool tok_ok = c.t0 + c.tw0 + tw < p.T;
        const int tl = tok_ok ? c.tw0 + tw : 0;
        float v[V];
#pragma unroll
        for (int j = 0; j < V; ++j) {
            const int e = min(s + j * S, E - 1);
            const float z = c.zs[tl * c.zstride + e];
            v[j] = j < vpl ? z : -INFINITY;
        }
        // with k <= kRegK every lane of the group keeps the picks in registers
        // (each pick goes to its slot by a select per slot, so no register is
        // indexed by the round); larger k use the pick area (every lane of the
        // group writes the same values)
        int* pk = c.area + tw * 32;
        float* pkv = (float*)(pk + 16);
        int hk[kRegK];
        float hv[kRegK];
#pragma unroll
        for (int j = 0; j < kRegK; ++j) {
            hk[j] = kNoPick;
            hv[j] = 0.f;
        }
        const bool regs = k <= kRegK;
        unsigned taken = dead;
        float prev = 0.f, top = 0.f, kth = 0.f;
        bool close = false;
        for (int r = 0; r < R; ++r) {
            // local arg-max in ascending expert order: strict > keeps the lower
            // index on ties; the first untaken slot is taken even at -inf
            float bv = -INFINITY;
            int be = kNoPick;
#pragma unroll
            for (int j = 0; j < V; ++j) {
                const bool t = !((taken >> j) & 1u) && (v[j] > bv || be == kNoPick);
                bv = t ? v[j] : bv;
                be = t ? key[j] : be;
            }
            group_argmax<S>(bv, be);
            const int e = pick_expert(be);
            if ((e & (S - 1)) == s) taken |= 1u << ((e / S) & 31);
            if (regs) {
#pragma unroll
                for (int j = 0; j < kRegK; ++j) {
                    hk[j] = r == j ? be : hk[j];
                    hv[j] = r == j ? bv : hv[j];
                }
            } else if (r < k) {
                pk[r] = be;
                pkv[r] = bv;
            }
            top = r == 0 ? bv : top;
            kth = r == k - 1 ? bv : kth;
            close = close || (r > 0 && prev - bv < kGap);
            prev = bv;
        }
        close = close && c.recheck;
        float se = 0.f;
#pragma unroll
        for (int j = 0; j < V; ++j) se += j < vpl ? __expf(v[j] - top) : 0.f;
        se = group_sum<S>(se);
        if (regs) finish_regs(p, c.t0 + tl, s, S, hk, hv, se, tok_ok && !close);
        else finish_token<float>(p, c.t0 + tl, s, S, pk, pkv, top, se, tok_ok && !close);
        if (tok_ok && close && s == 0) {
            const int pos = atomicAdd(c.fl_count, 1);
            c.fl_tok[pos] = tl;
            c.fl_thr[pos] = kth - kGap;
        }
    }
}

// Values per lane: the smallest of 1, 4, 16 that holds ceil(E / S). With S
// below 64 / TPW the group already spans all experts (V = 1); above it, S was
// raised because E needs more than 8 values per lane (V = 16).
template <int S, int TPW>
__device__ __forceinline__ void select_tokens_v(const RouteArgs& p, const SelectCtx& c, int lane) {
    constexpr int SB = kWave / TPW;
    const int vpl = (p.E + S - 1) / S;
    if constexpr (S < SB) {
        select_tokens<S, 1, TPW>(p, c, lane);
    } else if constexpr (S > SB) {
        select_tokens<S, 16, TPW>(p, c, lane);
    } else {
        if (vpl <= 1) select_tokens<S, 1, TPW>(p, c, lane);
        else if (vpl <= 4) select_tokens<S, 4, TPW>(p, c, lane);
        else if (vpl <= 8) select_tokens<S, 8, TPW>(p, c, lane);
        else select_tokens<S, 16, TPW>(p, c, lane);
    }
}

// Exact-product float64 dot products of one token row with up to 8 router rows
// over the 16-byte chunks [cb, ce) of the rows (ids[i] < 0: unused; the used
// ids come first). bf16 and fp32 products are exact in float64. Lane l takes
// the chunks cb+l, cb+l+64, ... (coalesced); a block of U chunks per lane is
// loaded together with the same chunks of every used router row, so a range of
// up to U*64 chunks costs one memory latency; each lane sums its chunks in
// order, then the wave reduces.
template <int MODE>
__device__ __forceinline__ void dot_f64_range(const char* xr, const char* w, size_t row_bytes, int cb, int ce,
                                              const int (&ids)[8], int lane, double (&out)[8]) {
    constexpr int U = 2;
    constexpr int EPC = mode_bf16(MODE) ? 8 : 4;  // elements per 16-byte chunk
    double acc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = 0.0;
    for (int c0 = cb; c0 < ce; c0 += kWave * U) {
        uint4 xv[U], wv[8][U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int c = c0 + u * kWave + lane;
            xv[u] = c < ce ? *(const uint4*)(xr + (size_t)c * 16) : make_uint4(0, 0, 0, 0);
#pragma unroll
            for (int i = 0; i < 8; ++i)
                wv[i][u] = (ids[i] >= 0 && c < ce) ? *(const uint4*)(w + (size_t)ids[i] * row_bytes + (size_t)c * 16)
                                                   : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if constexpr (mode_bf16(MODE)) {
                    const uint16_t* xs = (const uint16_t*)&xv[u];
                    const uint16_t* ws = (const uint16_t*)&wv[i][u];
#pragma unroll
                    for (int e = 0; e < EPC; ++e)
                        acc[i] += (double)bf16_to_f32(xs[e]) * (double)bf16_to_f32(ws[e]);
                } else {
                    const float* xs = (const float*)&xv[u];
                    const float* ws = (const float*)&wv[i][u];
#pragma unroll
                    for (int e = 0; e < EPC; ++e) acc[i] += (double)xs[e] * (double)ws[e];
                }
            }
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) out[i] = ids[i] >= 0 ? group_sum<kWave>(acc[i]) : 0.0;
}

// copies of super-chunk c into ring slot `slot` (padding copies go to the wave's dummy area)
template <class C>
__device__ __forceinline__ void route_issue(const uint16_t* const (&src)[C::DPW], const int (&lcol)[C::DPW],
                                            const uint32_t (&ldst)[C::DPW], const bool (&real)[C::DPW],
                                            uint32_t ring0, uint32_t dummy0, int d, int c, int slot) {
#pragma unroll
    for (int j = 0; j < C::DPW; ++j) {
        int col = c * C::KC + lcol[j];
        if (col >= d) col = 0;
        const uint32_t dst = real[j] ? ring0 + slot * C::SLOT + ldst[j] : dummy0;
        dma16(src[j] + col, __builtin_amdgcn_readfirstlane(dst));
    }
}

template <int TB, int NBLK, int KW>
__device__ __forceinline__ void logits_bf16(const RouteArgs& p, float* zs, char* ring, char* dummy, int t0) {
    using C = RouteCfg<TB, NBLK, KW>;
    const uint16_t* x = (const uint16_t*)p.x;
    const uint16_t* w = (const uint16_t*)p.w;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int tb = wave % TB, ks = wave / TB;
    const int q = lane >> 4, r16 = lane & 15;
    const int d = p.d, E = p.E, T = p.T;
    const int nsc = ceil_div(d, C::KC);
    const uint32_t ring0 = (uint32_t)(uintptr_t)ring;
    const uint32_t dummy0 = (uint32_t)(uintptr_t)dummy + wave * 1024;

    // per-lane copy sources of this wave's DMA instructions (column 0 of the super-chunk)
    const uint16_t* src[C::DPW];
    int lcol[C::DPW];      // logical column of this lane's chunk inside a super-chunk
    uint32_t ldst[C::DPW]; // LDS offset of the instruction inside a slot (or the dummy area)
    bool real[C::DPW];
    const int lrow = lane / C::CPR, lchk = lane % C::CPR;
#pragma unroll
    for (int j = 0; j < C::DPW; ++j) {
        const int g = wave + 4 * j;
        real[j] = g < C::TOT;
        if (g < C::XDMA) {
            const int rl = g * C::RPD + lrow;
            const int row = min(t0 + rl, T - 1);
            lcol[j] = (lchk ^ (rl & C::SWZ)) * 8;
            src[j] = x + (size_t)row * d;
            ldst[j] = g * C::RPD * C::ROWB;
        } else if (g < C::TOT) {
            const int rl = (g - C::XDMA) * C::RPD + lrow;
            const int row = min(rl, E - 1);
            lcol[j] = (lchk ^ (rl & C::SWZ)) * 8;
            src[j] = w + (size_t)row * d;
            ldst[j] = (C::BT + (g - C::XDMA) * C::RPD) * C::ROWB;
        } else {
            lcol[j] = 0;
            src[j] = x + (size_t)min(t0, T - 1) * d;
            ldst[j] = 0;
        }
    }
    f32x4 acc[NBLK];
#pragma unroll
    for (int nb = 0; nb < NBLK; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    // the bias of this lane's logit columns, in flight during the copies
    float bz[NBLK];
#pragma unroll
    for (int nb = 0; nb < NBLK; ++nb) {
        const int e = nb * 16 + r16;
        bz[nb] = (p.bias && e < E) ? p.bias[e] : 0.f;
    }
    const int arow = tb * 16 + r16;
    // logical chunks c0 .. c0+2KW-1 of this lane's A and B fragments: the k
    // index of MFMA u, lane group q, element j is chunk c0+u, element j
    constexpr int NU = 2 * KW;
    const int c0 = ks * 8 * KW + NU * q;
    int pa[NU], pb[NU];
#pragma unroll
    for (int u = 0; u < NU; ++u) {
        pa[u] = ((c0 + u) ^ (arow & C::SWZ)) << 4;
        pb[u] = ((c0 + u) ^ (r16 & C::SWZ)) << 4;
    }

    // prologue: super-chunks 0 .. NSLOT-2 in flight
#pragma unroll
    for (int c = 0; c < C::NSLOT - 1; ++c)
        if (c < nsc) route_issue<C>(src, lcol, ldst, real, ring0, dummy0, d, c, c);
    int slot = 0;
    for (int c = 0; c < nsc; ++c) {
        // copies issued so far: super-chunks 0 .. min(nsc-1, c+NSLOT-2)
        wait_vmcnt_rt<C::DPW>(min(nsc - 1 - c, C::NSLOT - 2));
        lds_reads_done();
        wg_barrier();
        // the slot read in the previous step is free for super-chunk c+NSLOT-1
        const int fill = c + C::NSLOT - 1;
        if (fill < nsc) route_issue<C>(src, lcol, ldst, real, ring0, dummy0, d, fill, slot == 0 ? C::NSLOT - 1 : slot - 1);
        const char* base = ring + slot * C::SLOT;
        const int col0 = c * C::KC + c0 * 8;
        uint4 a[NU];
#pragma unroll
        for (int u = 0; u < NU; ++u) {
            a[u] = *(const uint4*)(base + arow * C::ROWB + pa[u]);
            if (col0 + 8 * u >= d) a[u] = make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int u = 0; u < NU; ++u)
#pragma unroll
            for (int nb = 0; nb < NBLK; ++nb) {
                const char* bp = base + (C::BT + nb * 16 + r16) * C::ROWB;
                acc[nb] = mfma16(a[u], *(const uint4*)(bp + pb[u]), acc[nb]);
            }
        slot = slot + 1 == C::NSLOT ? 0 : slot + 1;
    }
    wait_vmcnt<0>();
    __syncthreads();

    // partial tiles of the d-split waves are summed in LDS (reusing the ring)
    float* part = (float*)ring;
    constexpr int BT = C::BT, EP = C::EP, KS = C::KS;
    if (KS > 1 && ks > 0) {
#pragma unroll
        for (int nb = 0; nb < NBLK; ++nb)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                part[((size_t)(ks - 1) * BT + tb * 16 + 4 * q + i) * EP + nb * 16 + r16] = acc[nb][i];
    }
    __syncthreads();
    if (ks == 0) {
#pragma unroll
        for (int nb = 0; nb < NBLK; ++nb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                float v = acc[nb][i];
                const int tl = tb * 16 + 4 * q + i;
                for (int kk = 1; kk < KS; ++kk) v += part[((size_t)(kk - 1) * BT + tl) * EP + nb * 16 + r16];
                const int e = nb * 16 + r16;
                if (e < E) zs[tl * (EP + 1) + e] = v + bz[nb];
            }
    }
}

// Logits of 16 tokens for E <= 8 and d = 1024 * NBAT, without barriers in
// the copy phase. Wave w owns the chunks [w*cq, w*cq + cq) of the d axis
// (16-byte chunks, cq = 32 * NBAT), taken in NBAT batches of 8 MFMAs. MFMA u
// of batch b covers chunks 32b + 4u .. 32b + 4u + 3 of the wave's range,
// lane group q taking chunk 32b + 4u + q of its token row (A) and of its
// router row (B): a k permutation that both operands share, under which a
// token row is read in 64-byte runs per load. The x tile goes straight from
// global memory into registers (all 8 * NBAT loads of a lane in flight at
// once); the wave's own columns of W_router (8 rows, rows past E repeat row
// E - 1) are copied into the wave's own LDS area before them, 4 KB per batch
// (row r, chunk j at slot 32r + (j ^ r): the eight rows a read phase touches
// fall in distinct banks), so a wave waits only for its own copies. The four
// partial tiles are summed in wave order.
// Batch B of the MFMAs of logits_bf16_res, then the following ones. The copies
// were issued before every x load: at most 8 * NBAT + 4 * (NBAT - 1 - B)
// operations in flight means the copies of batches 0..B have landed.
template <int NBAT, int B = 0>
__device__ __forceinline__ void res_mfma(const uint4 (&a)[NBAT][8], const char* wv, int nb, int q, f32x4& acc) {
    wait_vmcnt<8 * NBAT + 4 * (NBAT - 1 - B)>();
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        const uint4 bv = *(const uint4*)(wv + B * 4096 + (nb * 32 + ((4 * u + q) ^ nb)) * 16);
        acc = mfma16(a[B][u], bv, acc);
    }
    if constexpr (B + 1 < NBAT) res_mfma<NBAT, B + 1>(a, wv, nb, q, acc);
}

template <int NBAT>
__device__ __forceinline__ void logits_bf16_res(const RouteArgs& p, float* zs, char* wl, float* part, int t0) {
    const uint16_t* x = (const uint16_t*)p.x;
    const uint16_t* w = (const uint16_t*)p.w;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int q = lane >> 4, r16 = lane & 15;
    const int d = p.d, E = p.E, T = p.T;
    const int cb = wave * 32 * NBAT;
    // the bias of this lane's logit column, issued before every copy so that
    // the waits below cover it
    const float bz = (p.bias && r16 < E) ? p.bias[r16] : 0.f;
    char* wv = wl + wave * NBAT * 4096;
    const uint32_t wv0 = (uint32_t)(uintptr_t)wv;
    // 1. copies of the wave's router columns: instruction m of batch b fills
    // LDS rows 2m and 2m + 1 (lane i: row 2m + i / 32, slot i % 32)
    {
        const int j = lane & 31;
#pragma unroll
        for (int b = 0; b < NBAT; ++b)
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                const int r = 2 * m + (lane >> 5);
                const uint16_t* src = w + (size_t)min(r, E - 1) * d + (size_t)(cb + 32 * b + (j ^ r)) * 8;
                dma16(src, __builtin_amdgcn_readfirstlane(wv0 + (uint32_t)(b * 4096 + m * 1024)));
            }
    }
    // 2. the x tile of this lane: token t0 + r16 (clamped to the last token)
    const uint16_t* xr = x + (size_t)min(t0 + r16, T - 1) * d + (size_t)(cb + q) * 8;
    uint4 a[NBAT][8];
#pragma unroll
    for (int b = 0; b < NBAT; ++b)
#pragma unroll
        for (int u = 0; u < 8; ++u) a[b][u] = *(const uint4*)(xr + (size_t)(32 * b + 4 * u) * 8);
    // 3. MFMAs, batch by batch; B of lane (q, r16): LDS row r16 & 7
    f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
    res_mfma<NBAT>(a, wv, r16 & 7, q, acc);
    // 3. partial tiles: D[4q + i][r16] is token 4q + i, expert r16
    if (wave > 0) {
#pragma unroll
        for (int i = 0; i < 4; ++i) part[((wave - 1) * 16 + 4 * q + i) * 16 + r16] = acc[i];
    }
    __syncthreads();
    if (wave == 0 && r16 < E) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int tl = 4 * q + i;
            float v = acc[i];
#pragma unroll
            for (int kk = 0; kk < 3; ++kk) v += part[(kk * 16 + tl) * 16 + r16];
            zs[tl * 17 + r16] = v + bz;
        }
    }
}

// Logits of 32 tokens for 17..64 experts and d = 64 * NU. Wave w takes token
// block tb = w & 1 (16 tokens) and column half h = w >> 1; k-step u of a wave
// covers chunks 4u .. 4u + 3 of its half (16-byte chunks), lane group q taking
// chunk 4u + q of its token row (A) and of the router rows (B). The x tile
// goes straight into registers (NU loads per lane, all issued at once, after
// the first NS - 1 router slots); W_router alone streams through a ring of NS
// slots shared by the four waves, a slot holding 64 columns of each half of
// all 64 (padded) router rows: rows past E repeat row E - 1, slot row
// R = 64 h + e, its 8 chunks at positions chunk ^ (e & 7). The compiler waits
// for the whole x tile before the ring loop (a wait for one x load inside it
// would also wait for every copy issued after that load). The halves' partial
// tiles are summed in a fixed order.
template <int NU, int NS>
__device__ __forceinline__ void logits_bf16_xd(const RouteArgs& p, float* zs, char* ring, char* dummy, float* part,
                                               int t0) {
    constexpr int NSTEP = NU / 2;  // 64 columns of each half per ring step
    static_assert(NSTEP >= 1 && NS >= 2 && NS <= 8, "ring shape");
    const uint16_t* x = (const uint16_t*)p.x;
    const uint16_t* w = (const uint16_t*)p.w;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int q = lane >> 4, r16 = lane & 15;
    const int tb = wave & 1, h = wave >> 1;
    const int d = p.d, E = p.E, T = p.T;
    const int nchh = 4 * NU;  // chunks per half row
    float bz[4];
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
        const int e = nb * 16 + r16;
        bz[nb] = (p.bias && e < E) ? p.bias[e] : 0.f;
    }
    // copy instruction i = wave + 4j of a slot fills slot rows 8i .. 8i + 7
    // (lane: row 8i + lane / 8, position lane % 8); step c adds 64 columns
    const uint16_t* wsrc[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int R = 8 * (wave + 4 * j) + (lane >> 3);
        const int hh = R >> 6, e = R & 63;
        wsrc[j] = w + (size_t)min(e, E - 1) * d + (size_t)(hh * nchh + ((lane & 7) ^ (e & 7))) * 8;
    }
    // every workgroup of an XCD (workgroups are dealt to the 8 XCDs in turn)
    // first pulls its 1/32 share of W_router into that XCD's L2 (copies into
    // the wave's dummy area), so that the ring's copies hit in L2 instead of
    // all waiting on the same HBM misses step after step
    {
        const size_t wbytes = (size_t)E * d * 2;
        const size_t share = (wbytes / 32 + 4095) / 4096 * 4096;
        const size_t o0 = (size_t)((blockIdx.x >> 3) & 31) * share + (size_t)wave * (share / 4);
        const uint32_t dm = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)dummy + wave * 1024);
        for (size_t o = o0; o < o0 + share / 4 && o < wbytes; o += 1024)
            dma16((const char*)w + min(o + (size_t)lane * 16, wbytes - 16), dm);
    }
    const uint32_t ring0 = (uint32_t)(uintptr_t)ring;
    auto issue = [&](int c, int slot) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
            dma16(wsrc[j] + c * 64,
                  __builtin_amdgcn_readfirstlane(ring0 + (uint32_t)(slot * kXdSlot + (wave + 4 * j) * 1024)));
    };
#pragma unroll
    for (int c = 0; c < NS - 1; ++c)
        if (c < NSTEP) issue(c, c);
    const uint16_t* xr = x + (size_t)min(t0 + 16 * tb + r16, T - 1) * d + (size_t)(h * nchh + q) * 8;
    uint4 a[NU];
#pragma unroll
    for (int u = 0; u < NU; ++u) a[u] = *(const uint4*)(xr + u * 32);
#pragma unroll
    for (int u = 0; u < NU; ++u) asm volatile("" ::"v"(a[u].x), "v"(a[u].y), "v"(a[u].z), "v"(a[u].w));
    f32x4 acc[4];
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < NSTEP; ++c) {
        // copies issued so far: steps 0 .. min(NSTEP - 1, c + NS - 2)
        wait_vmcnt_rt<4>(min(NSTEP - 1 - c, NS - 2));
        wg_barrier();
        // the slot read in the previous step is free for step c + NS - 1
        if (c + NS - 1 < NSTEP) issue(c + NS - 1, (c + NS - 1) % NS);
        const char* base = ring + (c % NS) * kXdSlot;
#pragma unroll
        for (int uu = 0; uu < 2; ++uu) {
            const int j = 4 * uu + q;
#pragma unroll
            for (int nb = 0; nb < 4; ++nb) {
                const int e = nb * 16 + r16;
                const uint4 bv = *(const uint4*)(base + ((h * 64 + e) * 8 + (j ^ (e & 7))) * 16);
                acc[nb] = mfma16(a[2 * c + uu], bv, acc[nb]);
            }
        }
    }
    // D[4q + i][r16] of block nb: token 16 tb + 4q + i, expert 16 nb + r16
    if (h == 1) {
#pragma unroll
        for (int nb = 0; nb < 4; ++nb)
#pragma unroll
            for (int i = 0; i < 4; ++i) part[(tb * 16 + 4 * q + i) * 64 + nb * 16 + r16] = acc[nb][i];
    }
    __syncthreads();
    if (h == 0) {
#pragma unroll
        for (int nb = 0; nb < 4; ++nb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int tl = tb * 16 + 4 * q + i, e = nb * 16 + r16;
                if (e < E) zs[tl * 65 + e] = acc[nb][i] + part[tl * 64 + e] + bz[nb];
            }
    }
}

template <int MODE, int TB, int NBLK, int KW>
__global__ __launch_bounds__(kRouteThreads) void route_kernel(RouteArgs p) {
    extern __shared__ __align__(16) char smem[];
    const RouteSmem sm = route_smem<MODE, TB, NBLK, KW>(p.E, p.d);
    constexpr int BT = 16 * TB;
    constexpr int TPW = BT / 4;  // tokens per wave in the selection steps
    static_assert(TPW * 32 <= 512, "pick area of a wave");
    float* zs = (float*)smem;
    int* fl_count = (int*)(smem + sm.zs_bytes);
    int* fl_tok = fl_count + 4;
    float* fl_thr = (float*)(fl_tok + 4 * 16);
    char* dummy = smem + sm.zs_bytes + sm.flag_bytes + sm.cand_bytes;
    char* ring = dummy + sm.dummy_bytes;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    // per-wave area: picks of the wave's tokens (step 2), then candidate lists (step 3)
    int* cl = (int*)(smem + sm.zs_bytes + sm.flag_bytes) + wave * 512;
    const int t0 = blockIdx.x * BT;
    const int T = p.T, E = p.E, k = p.k;
    int* e2g_s = (int*)(smem + sm.zs_bytes + 1024);  // map, invalid entries -> -1
    if (tid < 4) fl_count[tid] = 0;
    // the map entry of expert tid (E <= the thread count), loaded before the
    // logits' copies are issued and written to LDS after them, so that its
    // latency does not delay the first copy
    const int g_in = tid < E ? p.e2g[tid] : -1;

    // ---- 1. logits tile
    if constexpr (MODE == MODE_BF16) {
        logits_bf16<TB, NBLK, KW>(p, zs, ring, dummy, t0);
    } else if constexpr (MODE == MODE_BF16_RES) {
        logits_bf16_res<KW>(p, zs, ring, (float*)(ring + res_w_bytes(p.d)), t0);
    } else if constexpr (MODE == MODE_BF16_XD) {
        logits_bf16_xd<xd_nu(KW), xd_ns(KW)>(p, zs, ring, dummy, (float*)(ring + xd_ns(KW) * kXdSlot), t0);
    } else if constexpr (MODE == MODE_F32) {
        const float* x = (const float*)p.x;
        const float* w = (const float*)p.w;
        for (int i = tid; i < BT * E; i += kRouteThreads) {
            int tl = i / E, e = i % E;
            int t = min(t0 + tl, T - 1);
            const float* xr = x + (size_t)t * p.d;
            const float* wr = w + (size_t)e * p.d;
            float acc = 0.f;
            for (int j = 0; j < p.d; ++j) acc = fmaf(xr[j], wr[j], acc);
            zs[tl * sm.zstride + e] = acc + (p.bias ? p.bias[e] : 0.f);
        }
    } else {
        for (int i = tid; i < BT * E; i += kRouteThreads) {
            int tl = i / E, e = i % E;
            int t = min(t0 + tl, T - 1);
            zs[tl * sm.zstride + e] = p.logits_in[(size_t)t * E + e];
        }
    }
    if (tid < E) e2g_s[tid] = (g_in >= 0 && g_in < p.G) ? g_in : -1;
    __syncthreads();
    if (p.logits_out) {
        for (int i = tid; i < BT * E; i += kRouteThreads) {
            int tl = i / E, e = i % E;
            if (t0 + tl < T) p.logits_out[(size_t)(t0 + tl) * E + e] = zs[tl * sm.zstride + e];
        }
    }

    // ---- 2. selection on the fp32 logits
    // A token occupies an aligned group of S lanes, S chosen so that the wave's
    // TPW tokens fill the wave in one pass where E allows (at most 16 values per
    // lane); lane s holds experts s, s+S, s+2S, ... .
    {
        int S = 1;
        while (S < E && S * TPW < kWave) S <<= 1;
        while (S * 16 < E) S <<= 1;
        SelectCtx c{zs, sm.zstride, cl, e2g_s, fl_count + wave, fl_tok + wave * 16, fl_thr + wave * 16,
                    t0, wave * TPW, MODE != MODE_LOGITS_IN};
        switch (S) {
            case 1: select_tokens_v<1, TPW>(p, c, lane); break;
            case 2: select_tokens_v<2, TPW>(p, c, lane); break;
            case 4: select_tokens_v<4, TPW>(p, c, lane); break;
            case 8: select_tokens_v<8, TPW>(p, c, lane); break;
            default: select_tokens_v<16, TPW>(p, c, lane); break;
        }
    }

    // ---- 3. float64 decision for the workgroup's queued tokens
    // Only experts whose fp32 logit is within the gap of the k-th value can be
    // in the exact top-k (the fp32 logits are far more accurate than the gap);
    // they are recomputed from exact float64 products and the picks are taken
    // among them. The queued tokens are spread over the four waves: a lone
    // token gets all four, two get two each, more get one each. The waves of a
    // team each sum the products of their share of the row into their own LDS
    // area; the team's first wave adds the shares in wave order and decides.
    if constexpr (MODE != MODE_LOGITS_IN) {
        __syncthreads();  // every wave's queue is complete
        const int q0 = fl_count[0], q1 = fl_count[1], q2 = fl_count[2], q3 = fl_count[3];
        const int nq = q0 + q1 + q2 + q3;
        const int sp = nq >= 3 ? 1 : (nq == 2 ? 2 : 4);  // waves per token
        const int team = wave / sp, mate = wave % sp;
        const size_t xrow_bytes = (size_t)p.d * (mode_bf16(MODE) ? 2 : 4);
        const int nch = (int)(xrow_bytes / 16);
        const int qc = ceil_div(nch, sp);
        const int cb = min(nch, mate * qc), ce = min(nch, cb + qc);
        // wave area: candidate ids [0, 1 KB), partial then exact logits of the
        // candidates (up to 32) at 1 KB, the pick list at 1280 B (16 packed
        // picks, 16 logits), the second buffer of partial logits at 1536 B
        int* pk3 = cl + 320;
        double* pv3 = (double*)(cl + 336);
        const int* area0 = (const int*)(smem + sm.zs_bytes + sm.flag_bytes);
        int parity = 0;
        for (int f0 = 0; f0 < nq; f0 += 4 / sp, parity ^= 1) {
            const int f = f0 + team;
            const bool active = f < nq;
            const int zoff = parity ? 384 : 256;  // int offset of this round's partials
            double* cz = (double*)(cl + zoff);
            int tl = 0;
            float thr = 0.f;
            if (active) {
                int qw = 0, pos = f;
                if (pos >= q0) {
                    pos -= q0;
                    qw = 1;
                    if (pos >= q1) {
                        pos -= q1;
                        qw = 2;
                        if (pos >= q2) {
                            pos -= q2;
                            qw = 3;
                        }
                    }
                }
                tl = fl_tok[qw * 16 + pos];
                thr = fl_thr[qw * 16 + pos];
            }
            const int t = t0 + tl;
            const char* xr = (const char*)p.x + (size_t)t * xrow_bytes;
            float fz[4];
            bool cand[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int e = lane + kWave * j;
                fz[j] = e < E ? zs[tl * sm.zstride + e] : -INFINITY;
                cand[j] = active && e < E && fz[j] >= thr;
            }
            // candidate list (ascending expert id): the waves of a team build
            // the same list, each in its own area
            int nc = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const unsigned long long m = __ballot(cand[j]);
                if (cand[j]) cl[nc + __popcll(m & ((1ull << lane) - 1ull))] = lane + kWave * j;
                nc += __popcll(m);
            }
            lds_reads_done();
            const bool shared = active && nc <= 32;
            // the deciding lane's bias, loaded before the products so that its
            // latency hides behind theirs
            const double bmid = (shared && mate == 0 && lane < nc && p.bias) ? (double)p.bias[cl[lane]] : 0.0;
            if (shared) {
                for (int b0 = 0; b0 < nc; b0 += 8) {
                    int ids[8];
                    double z[8];
#pragma unroll
                    for (int i = 0; i < 8; ++i) ids[i] = b0 + i < nc ? cl[b0 + i] : -1;
                    dot_f64_range<MODE>(xr, (const char*)p.w, xrow_bytes, cb, ce, ids, lane, z);
#pragma unroll
                    for (int i = 0; i < 8; ++i)
                        if (lane == i && ids[i] >= 0) cz[b0 + i] = z[i];
                }
            }
            // the shares of every team are complete; the partials of the next
            // round go to the other buffer, so one barrier per round suffices
            __syncthreads();
            if (!active || mate != 0) continue;
            double top;
            float sc = 0.f;  // this lane's softmax terms of candidates
            if (shared) {
                // lane i completes candidate i, then ranks it among all
                // candidates (ties: lower id); the ranks are a permutation, the
                // first k are the picks
                double mz = -INFINITY;
                int mid = 0;
                if (lane < nc) {
                    double zsum = 0.0;
                    for (int w = 0; w < sp; ++w) zsum += ((const double*)(area0 + (wave + w) * 512 + zoff))[lane];
                    mid = cl[lane];
                    mz = zsum + bmid;
                    cz[lane] = mz;
                }
                lds_reads_done();
                if (lane < nc) {
                    int rank = 0;
                    for (int j = 0; j < nc; ++j) rank += better(cz[j], cl[j], mz, mid) ? 1 : 0;
                    if (rank < k) {
                        pk3[rank] = pack_pick(mid, e2g_s, E);
                        pv3[rank] = mz;
                    }
                }
                lds_reads_done();
                top = pv3[0];
                if (lane < nc) sc = __expf((float)(mz - top));
            } else {
                // many near-equal logits: the team's first wave takes the whole
                // row alone, candidates stay in their experts' lanes
                double zz[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) zz[j] = -INFINITY;
                for (int b0 = 0; b0 < nc; b0 += 8) {
                    int ids[8];
#pragma unroll
                    for (int i = 0; i < 8; ++i) ids[i] = b0 + i < nc ? cl[b0 + i] : -1;
                    double z[8];
                    dot_f64_range<MODE>(xr, (const char*)p.w, xrow_bytes, 0, nch, ids, lane, z);
#pragma unroll
                    for (int i = 0; i < 8; ++i) {
                        if (ids[i] < 0) continue;
                        const double zi = z[i] + (p.bias ? (double)p.bias[ids[i]] : 0.0);
                        if (lane == (ids[i] & 63)) {
                            const int j = ids[i] >> 6;
                            if (j == 0) zz[0] = zi;
                            else if (j == 1) zz[1] = zi;
                            else if (j == 2) zz[2] = zi;
                            else zz[3] = zi;
                        }
                    }
                }
                unsigned taken = 0;
                for (int r = 0; r < k; ++r) {
                    double bv = -INFINITY;
                    int be = 0x7fffffff;
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const int e = lane + kWave * j;
                        if (cand[j] && !((taken >> j) & 1u) && better(zz[j], e, bv, be)) {
                            bv = zz[j];
                            be = e;
                        }
                    }
                    group_argmax<kWave>(bv, be);
                    if ((be & 63) == lane) taken |= 1u << (be >> 6);
                    if (lane == 0) {
                        pk3[r] = pack_pick(be, e2g_s, E);
                        pv3[r] = bv;
                    }
                }
                lds_reads_done();
                top = pv3[0];
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (cand[j]) sc += __expf((float)(zz[j] - top));
            }
            // the other experts' softmax terms from their fp32 logits
            float so = sc;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int e = lane + kWave * j;
                if (e < E && !cand[j]) so += __expf((float)((double)fz[j] - top));
            }
            so = group_sum<kWave>(so);
            if (k <= kRegK) {
                // the pick list into registers (entries past k are never used)
                int hk[kRegK];
                double hv[kRegK];
#pragma unroll
                for (int j = 0; j < kRegK; ++j) {
                    hk[j] = pk3[j];
                    hv[j] = pv3[j];
                }
                finish_regs(p, t, lane, kWave, hk, hv, so, true);
            } else {
                finish_token<double>(p, t, lane, kWave, pk3, pv3, top, so, true);
            }
            lds_reads_done();  // cl is rewritten for the next queued token
        }
    }
}

template <int MODE, int TB, int NBLK, int KW = 1>
hipError_t launch_one(const RouteArgs& a, hipStream_t s) {
    const RouteSmem sm = route_smem<MODE, TB, NBLK, KW>(a.E, a.d);
    auto kern = route_kernel<MODE, TB, NBLK, KW>;
    // the kernel's dynamic LDS limit is raised to the whole 160 KiB once per
    // device (the attribute only permits; each launch asks for what it uses)
    static std::atomic<uint32_t> raised{0};  // bit d: done on device d < 32
    int dev = 0;
    hipError_t err = hipGetDevice(&dev);
    if (err != hipSuccess) return err;
    const uint32_t bit = dev >= 0 && dev < 32 ? 1u << dev : 0u;
    if (bit == 0u || !(raised.load(std::memory_order_acquire) & bit)) {
        err = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
        if (err != hipSuccess) return err;
        raised.fetch_or(bit, std::memory_order_release);
    }
    dim3 grid(ceil_div(a.T, 16 * TB));
    hipLaunchKernelGGL(kern, grid, dim3(kRouteThreads), sm.total(), s, a);
    return hipGetLastError();
}

// x straight into registers, 16 tokens per workgroup: E <= 8 and d a whole
// number (at most 4) of 1024-column batches per wave
bool res_fits(const RouteArgs& a) { return a.E <= 8 && a.d % 1024 == 0 && a.d <= 4096; }
hipError_t launch_res(const RouteArgs& a, hipStream_t s) {
    switch (a.d / 1024) {
        case 1: return launch_one<MODE_BF16_RES, 1, 1, 1>(a, s);
        case 2: return launch_one<MODE_BF16_RES, 1, 1, 2>(a, s);
        case 3: return launch_one<MODE_BF16_RES, 1, 1, 3>(a, s);
        default: return launch_one<MODE_BF16_RES, 1, 1, 4>(a, s);
    }
}

// x straight into registers, W_router alone through the ring: 17..64 experts,
// d of 512, 1024 or 2048 columns, at least 4096 tokens (128 workgroups of 32
// tokens); more than 256 workgroups run two per CU, with three slots each
bool xd_fits(const RouteArgs& a) {
    return a.E > 16 && a.E <= 64 && (a.d == 512 || a.d == 1024 || a.d == 2048) && a.T >= 4096;
}
template <int NU>
hipError_t launch_xd_nu(const RouteArgs& a, hipStream_t s) {
    if (ceil_div(a.T, 32) > 256) return launch_one<MODE_BF16_XD, 2, 4, NU + 64 * 3>(a, s);
    return launch_one<MODE_BF16_XD, 2, 4, NU + 64 * 6>(a, s);
}
hipError_t launch_xd(const RouteArgs& a, hipStream_t s) {
    if (a.d == 2048) return launch_xd_nu<32>(a, s);
    if (a.d == 1024) return launch_xd_nu<16>(a, s);
    return launch_xd_nu<8>(a, s);
}

template <int TB>
hipError_t launch_bf16(const RouteArgs& a, hipStream_t s) {
    // two 64-column units per wave and copy step where two ring slots still
    // fit (fewer barriers per byte); tiles of 16 or 32 tokens with up to 64
    // experts keep one (32 tokens: five 24 KB slots instead of two 48 KB
    // ones, measured 4 % faster warm and 8 % cold on 8192 tokens)
    if (a.E <= 16) return launch_one<MODE_BF16, TB, 1, 2>(a, s);
    if constexpr (TB > 2) {
        if (a.E <= 64) return launch_one<MODE_BF16, TB, 4, 2>(a, s);
    } else {
        if (a.E <= 64) return launch_one<MODE_BF16, TB, 4, 1>(a, s);
    }
    return launch_one<MODE_BF16, 4, 16>(a, s);
}

}  // namespace

hipError_t launch_route(const RouteArgs& a, hipStream_t s) {
    if (a.T == 0) return hipSuccess;
    if (a.logits_in) return launch_one<MODE_LOGITS_IN, 1, 1>(a, s);
    if (a.dtype == BMOE_F32) return launch_one<MODE_F32, 1, 1>(a, s);
    if (res_fits(a)) return launch_res(a, s);
    if (xd_fits(a)) return launch_xd(a, s);
    // tokens per workgroup: as many as keep >= 256 workgroups (one per CU), so
    // that W_router (L2-resident) is re-read as few times as possible
    if (a.T >= 64 * 256) return launch_bf16<4>(a, s);
    if (a.T >= 32 * 256) return launch_bf16<2>(a, s);
    return launch_bf16<1>(a, s);
}

}  // namespace bmoe
