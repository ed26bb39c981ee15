// Gate and united-expert substitution (paper Sec. 2.1 gating, Eq. 2 map,
// Sec. 4.3 closing paragraph: the gate picks experts, the map replaces them).
//
// One workgroup (4 waves) owns BT = 16*TB tokens:
//   1. logits tile [BT, E] into LDS:
//        bf16: x rows stream from HBM straight into MFMA A-fragments; W_router
//              is staged through LDS in super-chunks of KS*64 columns (double
//              buffered) and shared by the 4 waves; 16x16x32 bf16 MFMA, fp32
//              accumulate; with KS > 1 the waves split the d axis and their
//              partial tiles are summed in LDS in a fixed order;
//        f32:  one (token, expert) dot product per thread;
//        logits_in: copied.
//   2. per token, a segment of S = pow2ceil(E) lanes (<= 64) holds the E logits;
//      k+1 rounds of segment arg-max by xor-shuffles give the picks in order
//      (ties: lower expert index). If two adjacent values among the top (k+1)
//      are closer than BMOE_ROUTE_RECHECK_GAP the token is queued for step 3.
//      Otherwise softmax, optional renormalisation, the map and the per-group
//      merge are done by the k slot lanes and written out.
//   3. a queued token is decided again in float64: every expert whose fp32 logit
//      is within the gap of the k-th value is recomputed from exact float64
//      products (a whole wave per expert), and the top-k is picked among those.
#include "bmoe_common.h"

namespace bmoe {
namespace {

constexpr int kRouteThreads = 256;
constexpr float kGap = BMOE_ROUTE_RECHECK_GAP;
constexpr int kMaxK = BMOE_MAX_TOPK;

enum { MODE_LOGITS_IN = 0, MODE_F32 = 1, MODE_BF16 = 2 };

struct RouteSmem {
    int bt, zstride, e_pad, ks;
    size_t zs_bytes, flag_bytes, wbuf_bytes;
    __host__ __device__ size_t total() const { return zs_bytes + flag_bytes + wbuf_bytes; }
};

__host__ __device__ inline RouteSmem route_smem(int mode, int tb, int nblk, int E) {
    RouteSmem s;
    s.bt = 16 * tb;
    s.e_pad = (mode == MODE_BF16) ? 16 * nblk : ((E + 15) / 16) * 16;
    s.zstride = s.e_pad + 1;
    s.ks = 4 / tb;
    s.zs_bytes = ((size_t)s.bt * s.zstride * 4 + 15) / 16 * 16;
    s.flag_bytes = 1024;
    s.wbuf_bytes = (mode == MODE_BF16) ? (size_t)2 * s.e_pad * (s.ks * 64 + 8) * 2 : 0;
    return s;
}

__device__ __forceinline__ bool better(float v, int e, float bv, int be) {
    return v > bv || (v == bv && e < be);
}
__device__ __forceinline__ bool better(double v, int e, double bv, int be) {
    return v > bv || (v == bv && e < be);
}

template <typename V>
__device__ __forceinline__ void seg_argmax(V& bv, int& be, int S) {
    for (int off = 1; off < S; off <<= 1) {
        V ov = __shfl_xor(bv, off);
        int oe = __shfl_xor(be, off);
        if (better(ov, oe, bv, be)) { bv = ov; be = oe; }
    }
}

template <typename V>
__device__ __forceinline__ V seg_sum(V v, int S) {
    for (int off = 1; off < S; off <<= 1) v += __shfl_xor(v, off);
    return v;
}

// Softmax weight, renormalisation, map and merge for the k slot lanes of a
// segment; lane s (< k) holds pick s. Writes the token's outputs.
template <typename V>
__device__ __forceinline__ void finish_token(const RouteArgs& p, int t, int s, int S, int pick,
                                             V pick_val, V top, V sum_exp, bool write) {
    const int k = p.k;
    float w = 0.f;
    if (s < k) {
        if constexpr (sizeof(V) == 8) w = (float)(exp(pick_val - top) / sum_exp);
        else w = expf(pick_val - top) / sum_exp;
    }
    if (p.norm) {
        float tot = seg_sum(s < k ? w : 0.f, S);
        w = w / tot;
    }
    int g = (s < k) ? p.e2g[pick] : -2;
    if (s < k && (g < 0 || g >= p.G)) g = -1;  // unvalidated map entry: no call
    bool dup = false;
    float gate = 0.f;
    for (int j = 0; j < k; ++j) {
        int gj = __shfl(g, j, S);
        float wj = __shfl(w, j, S);
        if (j < s && gj == g) dup = true;
        if (j >= s && gj == g) gate += wj;
    }
    if (write && s < k) {
        size_t o = (size_t)t * k + s;
        p.topk_idx[o] = pick;
        p.topk_w[o] = w;
        bool valid = !dup && g >= 0;
        p.slot_group[o] = valid ? g : -1;
        p.slot_gate[o] = valid ? gate : 0.f;
    }
}

// Exact-product float64 dot product of one token row and one router row;
// every lane of the wave takes 8-element chunks; the result is in all lanes.
template <int MODE>
__device__ __forceinline__ double dot_f64(const void* xr, const void* wr, int d, int lane) {
    double acc = 0.0;
    const int nch = d / 8;
    for (int c = lane; c < nch; c += kWave) {
        if constexpr (MODE == MODE_BF16) {
            uint4 xv = *((const uint4*)xr + c);
            uint4 wv = *((const uint4*)wr + c);
            const uint16_t* xs = (const uint16_t*)&xv;
            const uint16_t* ws = (const uint16_t*)&wv;
#pragma unroll
            for (int i = 0; i < 8; ++i) acc += (double)bf16_to_f32(xs[i]) * (double)bf16_to_f32(ws[i]);
        } else {
            const float4* xf = (const float4*)xr + 2 * c;
            const float4* wf = (const float4*)wr + 2 * c;
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                float4 a = xf[h], b = wf[h];
                acc += (double)a.x * (double)b.x;
                acc += (double)a.y * (double)b.y;
                acc += (double)a.z * (double)b.z;
                acc += (double)a.w * (double)b.w;
            }
        }
    }
    return seg_sum(acc, kWave);
}

template <int WPT, int KC, int WCH>
__device__ __forceinline__ void route_load_w(uint4 (&wreg)[WPT], const uint16_t* w, int E, int d,
                                             int c, int tid) {
#pragma unroll
    for (int i = 0; i < WPT; ++i) {
        int idx = tid + kRouteThreads * i;
        int er = idx / (KC / 8), cc = idx % (KC / 8);
        int col = c * KC + cc * 8;
        wreg[i] = (idx < WCH && er < E && col < d) ? *(const uint4*)(w + (size_t)er * d + col)
                                                   : make_uint4(0, 0, 0, 0);
    }
}

template <int WPT, int KC, int WCH, int EP, int WROW>
__device__ __forceinline__ void route_store_w(const uint4 (&wreg)[WPT], uint16_t* wb, int buf, int tid) {
#pragma unroll
    for (int i = 0; i < WPT; ++i) {
        int idx = tid + kRouteThreads * i;
        if (idx < WCH) {
            int er = idx / (KC / 8), cc = idx % (KC / 8);
            *(uint4*)(wb + ((size_t)buf * EP + er) * WROW + cc * 8) = wreg[i];
        }
    }
}

template <int KC>
__device__ __forceinline__ void route_load_a(const uint16_t* xr, int d, int c, int ks, int q,
                                             uint4& a0, uint4& a1) {
    int col = c * KC + ks * 64 + 16 * q;
    a0 = col < d ? *(const uint4*)(xr + col) : make_uint4(0, 0, 0, 0);
    a1 = col + 8 < d ? *(const uint4*)(xr + col + 8) : make_uint4(0, 0, 0, 0);
}

template <int TB, int NBLK>
__device__ __forceinline__ void logits_bf16(const RouteArgs& p, const RouteSmem& sm, float* zs,
                                            char* wraw, int t0) {
    constexpr int KS = 4 / TB;
    constexpr int KC = KS * 64;
    constexpr int WROW = KC + 8;
    constexpr int EP = NBLK * 16;
    constexpr int WCH = EP * KC / 8;                 // 16-byte chunks per super-chunk
    constexpr int WPT = (WCH + kRouteThreads - 1) / kRouteThreads;
    const uint16_t* x = (const uint16_t*)p.x;
    const uint16_t* w = (const uint16_t*)p.w;
    uint16_t* wb = (uint16_t*)wraw;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int tb = wave % TB, ks = wave / TB;
    const int q = lane >> 4, r16 = lane & 15;
    const int d = p.d, E = p.E;
    int row = t0 + tb * 16 + r16;
    if (row > p.T - 1) row = p.T - 1;
    const uint16_t* xr = x + (size_t)row * d;
    const int nsc = ceil_div(d, KC);
    const uint4 zero = make_uint4(0, 0, 0, 0);

    uint4 wreg[WPT];
    f32x4 acc[NBLK];
#pragma unroll
    for (int nb = 0; nb < NBLK; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};

    uint4 a0, a1;
    route_load_w<WPT, KC, WCH>(wreg, w, E, d, 0, tid);
    route_load_a<KC>(xr, d, 0, ks, q, a0, a1);
    route_store_w<WPT, KC, WCH, EP, WROW>(wreg, wb, 0, tid);
    __syncthreads();
    for (int c = 0; c < nsc; ++c) {
        uint4 n0 = zero, n1 = zero;
        const bool more = c + 1 < nsc;
        if (more) {
            route_load_w<WPT, KC, WCH>(wreg, w, E, d, c + 1, tid);
            route_load_a<KC>(xr, d, c + 1, ks, q, n0, n1);
        }
        const uint16_t* wbc = wb + (size_t)(c & 1) * EP * WROW;
#pragma unroll
        for (int nb = 0; nb < NBLK; ++nb) {
            const uint16_t* bp = wbc + (nb * 16 + r16) * WROW + ks * 64 + 16 * q;
            uint4 b0 = *(const uint4*)bp;
            uint4 b1 = *(const uint4*)(bp + 8);
            acc[nb] = mfma16(a0, b0, acc[nb]);
            acc[nb] = mfma16(a1, b1, acc[nb]);
        }
        if (more) {
            route_store_w<WPT, KC, WCH, EP, WROW>(wreg, wb, (c + 1) & 1, tid);
            a0 = n0;
            a1 = n1;
        }
        __syncthreads();
    }

    // partial tiles of the d-split waves are summed in LDS (reusing the W buffer)
    float* part = (float*)wraw;
    const int BT = 16 * TB;
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
                if (e < E) zs[tl * sm.zstride + e] = v + (p.bias ? p.bias[e] : 0.f);
            }
    }
}

template <int MODE, int TB, int NBLK>
__global__ __launch_bounds__(kRouteThreads) void route_kernel(RouteArgs p) {
    extern __shared__ __align__(16) char smem[];
    const RouteSmem sm = route_smem(MODE, TB, NBLK, p.E);
    constexpr int BT = 16 * TB;
    constexpr int TPW = BT / 4;  // tokens per wave in the selection steps
    float* zs = (float*)smem;
    int* fl_count = (int*)(smem + sm.zs_bytes);
    int* fl_tok = fl_count + 4;
    float* fl_thr = (float*)(fl_tok + 4 * 16);
    char* wraw = smem + sm.zs_bytes + sm.flag_bytes;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int t0 = blockIdx.x * BT;
    const int T = p.T, E = p.E, k = p.k;
    if (tid < 4) fl_count[tid] = 0;

    // ---- 1. logits tile
    if constexpr (MODE == MODE_BF16) {
        logits_bf16<TB, NBLK>(p, sm, zs, wraw, t0);
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
    __syncthreads();
    if (p.logits_out) {
        for (int i = tid; i < BT * E; i += kRouteThreads) {
            int tl = i / E, e = i % E;
            if (t0 + tl < T) p.logits_out[(size_t)(t0 + tl) * E + e] = zs[tl * sm.zstride + e];
        }
    }

    // ---- 2. selection on the fp32 logits
    int S = 1;
    while (S < E && S < 64) S <<= 1;
    const int VPL = ceil_div(E, S);
    const int P = kWave / S;
    const int s = lane % S, seg = lane / S;
    const int R = min(k + 1, E);
    const bool recheck = (MODE != MODE_LOGITS_IN);
    for (int base = 0; base < TPW; base += P) {
        const int tw = base + seg;
        const bool tok_ok = tw < TPW && t0 + wave * TPW + tw < T;
        const int tl = tok_ok ? wave * TPW + tw : 0;
        float v[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            int e = s + S * j;
            v[j] = (j < VPL && e < E) ? zs[tl * sm.zstride + e] : -INFINITY;
        }
        unsigned taken = 0;
        float prev = 0.f, top = 0.f, kth = 0.f, my_val = 0.f;
        int my_pick = 0;
        bool close = false;
        for (int r = 0; r < R; ++r) {
            float bv = -INFINITY;
            int be = 0x7fffffff;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                int e = s + S * j;
                if (j < VPL && e < E && !((taken >> j) & 1u) && better(v[j], e, bv, be)) {
                    bv = v[j];
                    be = e;
                }
            }
            seg_argmax(bv, be, S);
            if (be % S == s) taken |= 1u << (be / S);
            if (s == r) { my_pick = be; my_val = bv; }
            if (r == 0) top = bv;
            if (r == k - 1) kth = bv;
            if (r > 0 && prev - bv < kGap) close = true;
            prev = bv;
        }
        close = close && recheck;
        float se = 0.f;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            int e = s + S * j;
            if (j < VPL && e < E) se += expf(v[j] - top);
        }
        se = seg_sum(se, S);
        finish_token<float>(p, t0 + tl, s, S, my_pick, my_val, top, se, tok_ok && !close);
        if (tok_ok && close && s == 0) {
            int pos = atomicAdd(&fl_count[wave], 1);
            fl_tok[wave * 16 + pos] = tl;
            fl_thr[wave * 16 + pos] = kth - kGap;
        }
    }
    __syncthreads();

    // ---- 3. float64 decision for queued tokens (one wave per token)
    if constexpr (MODE != MODE_LOGITS_IN) {
        const int nf = fl_count[wave];
        const size_t xrow_bytes = (size_t)p.d * (MODE == MODE_BF16 ? 2 : 4);
        for (int f = 0; f < nf; ++f) {
            const int tl = fl_tok[wave * 16 + f];
            const float thr = fl_thr[wave * 16 + f];
            const int t = t0 + tl;
            const char* xr = (const char*)p.x + (size_t)t * xrow_bytes;
            double zz[4];
            float fz[4];
            bool cand[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                int e = lane + kWave * j;
                fz[j] = e < E ? zs[tl * sm.zstride + e] : -INFINITY;
                cand[j] = e < E && fz[j] >= thr;
                zz[j] = -INFINITY;
            }
            unsigned long long mk[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) mk[j] = __ballot(cand[j]);
            for (int j = 0; j < 4; ++j) {
                unsigned long long m = j == 0 ? mk[0] : j == 1 ? mk[1] : j == 2 ? mk[2] : mk[3];
                while (m) {
                    const int b = __ffsll((long long)m) - 1;
                    m &= m - 1;
                    const int e = b + kWave * j;
                    double z = dot_f64<MODE>(xr, (const char*)p.w + (size_t)e * xrow_bytes, p.d, lane);
                    if (p.bias) z += (double)p.bias[e];
                    if (lane == b) {
                        if (j == 0) zz[0] = z;
                        else if (j == 1) zz[1] = z;
                        else if (j == 2) zz[2] = z;
                        else zz[3] = z;
                    }
                }
            }
            unsigned taken = 0;
            double top = 0.0, my_val = 0.0;
            int my_pick = 0;
            for (int r = 0; r < k; ++r) {
                double bv = -INFINITY;
                int be = 0x7fffffff;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    int e = lane + kWave * j;
                    if (cand[j] && !((taken >> j) & 1u) && better(zz[j], e, bv, be)) {
                        bv = zz[j];
                        be = e;
                    }
                }
                seg_argmax(bv, be, kWave);
                if ((be & 63) == lane) taken |= 1u << (be >> 6);
                if (lane == r) { my_pick = be; my_val = bv; }
                if (r == 0) top = bv;
            }
            double se = 0.0;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                int e = lane + kWave * j;
                if (e < E) se += exp((cand[j] ? zz[j] : (double)fz[j]) - top);
            }
            se = seg_sum(se, kWave);
            finish_token<double>(p, t, lane, kWave, my_pick, my_val, top, se, true);
        }
    }
}

template <int MODE, int TB, int NBLK>
hipError_t launch_one(const RouteArgs& a, hipStream_t s) {
    const RouteSmem sm = route_smem(MODE, TB, NBLK, a.E);
    auto kern = route_kernel<MODE, TB, NBLK>;
    hipError_t err = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize,
                                         (int)sm.total());
    if (err != hipSuccess) return err;
    dim3 grid(ceil_div(a.T, 16 * TB));
    hipLaunchKernelGGL(kern, grid, dim3(kRouteThreads), sm.total(), s, a);
    return hipGetLastError();
}

template <int TB>
hipError_t launch_bf16(const RouteArgs& a, hipStream_t s) {
    if (a.E <= 16) return launch_one<MODE_BF16, TB, 1>(a, s);
    if (a.E <= 64) return launch_one<MODE_BF16, TB, 4>(a, s);
    return launch_one<MODE_BF16, 4, 16>(a, s);
}

}  // namespace

hipError_t launch_route(const RouteArgs& a, hipStream_t s) {
    if (a.T == 0) return hipSuccess;
    if (a.logits_in) return launch_one<MODE_LOGITS_IN, 1, 1>(a, s);
    if (a.dtype == BMOE_F32) return launch_one<MODE_F32, 1, 1>(a, s);
    // tokens per workgroup: as many as keep >= 256 workgroups (one per CU), so
    // that W_router (L2-resident) is re-read as few times as possible
    if (a.T >= 64 * 256) return launch_bf16<4>(a, s);
    if (a.T >= 32 * 256) return launch_bf16<2>(a, s);
    return launch_bf16<1>(a, s);
}

}  // namespace bmoe
