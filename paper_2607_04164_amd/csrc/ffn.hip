// Grouped SwiGLU FFN over the united experts (each expert an FFN of Sec. 2.1;
// SwiGLU form): for the rows of segment s,
//   h = silu(A W_gate[s]^T) * (A W_up[s]^T)     (gate/up fused, one pass over A)
//   y = h W_down[s]^T
//
// bf16 path: one grouped-GEMM kernel template, 256 threads (4 waves, 2x2),
// 32x32x16 bf16 MFMA with fp32 accumulation, A and B tiles double-buffered in
// LDS with padded rows (conflict-free 128-bit fragment reads), global loads of
// the next K-step in flight while the current one runs on the matrix cores.
//   gate/up: BM=128, BN=128 columns of BOTH W_gate and W_up (each wave 64x64 of
//            each), epilogue silu(g)*u -> bf16 h;
//   down:    BM=128, BN=256 (each wave 64x128), epilogue -> bf16 y.
// Both epilogues stage the tile through LDS and store 128-bit row chunks.
// Tile schedule without a host sync: the grid covers the worst case
// (ceil(rows_cap/BM) + n_seg M-tiles times the N-tiles); every workgroup
// rebuilds the per-segment M-tile prefix from the device offsets, maps its
// (XCD-swizzled) id to (segment, N-tile, M-tile) with M fastest, so the
// M-tiles that share a weight panel run together on one XCD, and workgroups
// past the real tile count exit at once.
//
// f32 path (small correctness configurations): one output element per thread.
#include "bmoe_common.h"

namespace bmoe {
namespace {

constexpr int kGemmThreads = 256;

struct GemmParams {
    const uint16_t* A;
    const uint16_t* B0;
    const uint16_t* B1;
    uint16_t* C;
    const int32_t* offsets;
    int n_seg, rows_cap, N, K;
};

template <bool GATED, int BM, int BN, int BK>
struct GemmCfg {
    static constexpr int WM = 2, WN = 2;
    static constexpr int WTM = BM / WM, WTN = BN / WN;
    static constexpr int MB = WTM / 32, NB = WTN / 32;
    static constexpr int NMAT = GATED ? 2 : 1;
    static constexpr int LROW = BK + 8;  // padded LDS row (elements)
    static constexpr int KCH = BK / 8;   // 16-byte chunks per tile row
    static constexpr int A_CH = BM * KCH / kGemmThreads;
    static constexpr int B_CH = BN * KCH / kGemmThreads;
    static constexpr int A_BYTES = 2 * BM * LROW * 2;
    static constexpr int B_BYTES = 2 * BN * LROW * 2;
    static constexpr int SROW = WTN + 8;  // epilogue staging row (elements)
    static constexpr int STAGE_BYTES = 4 * WTM * SROW * 2;
    static constexpr int MAIN_BYTES = A_BYTES + NMAT * B_BYTES;
    static constexpr int SMEM = MAIN_BYTES > STAGE_BYTES ? MAIN_BYTES : STAGE_BYTES;
    static_assert(BM * KCH % kGemmThreads == 0 && BN * KCH % kGemmThreads == 0, "tile/threads");
};

__device__ __forceinline__ int xcd_swizzle(int b, int nblocks) {
    // workgroups are dealt to the 8 XCDs round-robin; give each XCD a
    // contiguous range of logical tiles (nblocks is a multiple of 8)
    const int per = nblocks >> 3;
    return (b & 7) * per + (b >> 3);
}

template <class C>
__device__ __forceinline__ void gemm_gload(uint4 (&ra)[C::A_CH], uint4 (&rb)[C::NMAT][C::B_CH],
                                           const uint16_t* A, const uint16_t* B0, const uint16_t* B1,
                                           int tid, int k0, int m0, int m_end, int n0, int N, int K) {
#pragma unroll
    for (int i = 0; i < C::A_CH; ++i) {
        const int c = tid + kGemmThreads * i;
        const int r = c / C::KCH, cc = c % C::KCH;
        const int gm = min(m0 + r, m_end - 1);
        const int gk = k0 + cc * 8;
        ra[i] = gk < K ? *(const uint4*)(A + (size_t)gm * K + gk) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int mat = 0; mat < C::NMAT; ++mat) {
        const uint16_t* B = mat == 0 ? B0 : B1;
#pragma unroll
        for (int i = 0; i < C::B_CH; ++i) {
            const int c = tid + kGemmThreads * i;
            const int r = c / C::KCH, cc = c % C::KCH;
            const int gn = min(n0 + r, N - 1);
            const int gk = k0 + cc * 8;
            rb[mat][i] = gk < K ? *(const uint4*)(B + (size_t)gn * K + gk) : make_uint4(0, 0, 0, 0);
        }
    }
}

template <class C>
__device__ __forceinline__ void gemm_sstore(const uint4 (&ra)[C::A_CH], const uint4 (&rb)[C::NMAT][C::B_CH],
                                            uint16_t* sA, uint16_t* sB, int tid, int buf) {
    constexpr int BM = C::A_CH * kGemmThreads / C::KCH;
    constexpr int BN = C::B_CH * kGemmThreads / C::KCH;
#pragma unroll
    for (int i = 0; i < C::A_CH; ++i) {
        const int c = tid + kGemmThreads * i;
        const int r = c / C::KCH, cc = c % C::KCH;
        *(uint4*)(sA + (size_t)(buf * BM + r) * C::LROW + cc * 8) = ra[i];
    }
#pragma unroll
    for (int mat = 0; mat < C::NMAT; ++mat)
#pragma unroll
        for (int i = 0; i < C::B_CH; ++i) {
            const int c = tid + kGemmThreads * i;
            const int r = c / C::KCH, cc = c % C::KCH;
            *(uint4*)(sB + (size_t)((mat * 2 + buf) * BN + r) * C::LROW + cc * 8) = rb[mat][i];
        }
}

template <bool GATED, int BM, int BN, int BK>
__global__ __launch_bounds__(kGemmThreads, 1) void grouped_gemm_kernel(GemmParams p) {
    using C = GemmCfg<GATED, BM, BN, BK>;
    __shared__ __align__(16) char smem[C::SMEM];
    __shared__ int s_scan[256];
    __shared__ int s_mt[BMOE_MAX_EXPERTS + 1];
    __shared__ int s_beg[BMOE_MAX_EXPERTS];
    __shared__ int s_end[BMOE_MAX_EXPERTS];

    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int n_seg = p.n_seg, N = p.N, K = p.K;

    // ---- tile schedule from the device offsets
    int cnt = 0;
    if (tid < n_seg) {
        int beg = min(max(p.offsets[tid], 0), p.rows_cap);
        int end = min(max(p.offsets[tid + 1], beg), p.rows_cap);
        s_beg[tid] = beg;
        s_end[tid] = end;
        cnt = ceil_div(end - beg, BM);
    }
    int total_mt;
    const int ex = block_exclusive_scan_256(cnt, s_scan, &total_mt);
    if (tid < n_seg) s_mt[tid] = ex;
    if (tid == 0) s_mt[n_seg] = total_mt;
    __syncthreads();
    const int NT = ceil_div(N, BN);
    const int L = xcd_swizzle(blockIdx.x, gridDim.x);
    if (L >= total_mt * NT) return;
    int lo = 0, hi = n_seg - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (s_mt[mid] * NT <= L) lo = mid;
        else hi = mid - 1;
    }
    const int s = lo;
    const int mts = s_mt[s + 1] - s_mt[s];
    const int local = L - s_mt[s] * NT;
    const int nt = local / mts, mt = local % mts;
    const int m0 = s_beg[s] + mt * BM, m_end = s_end[s];
    const int n0 = nt * BN;

    uint16_t* sA = (uint16_t*)smem;
    uint16_t* sB = (uint16_t*)(smem + C::A_BYTES);
    const uint16_t* Bm[2] = {p.B0 + (size_t)s * N * K, GATED ? p.B1 + (size_t)s * N * K : p.B0};

    // global -> register staging of one K-step
    uint4 ra[C::A_CH];
    uint4 rb[C::NMAT][C::B_CH];
    f32x16 acc[C::NMAT][C::MB][C::NB];
#pragma unroll
    for (int mat = 0; mat < C::NMAT; ++mat)
#pragma unroll
        for (int mb = 0; mb < C::MB; ++mb)
#pragma unroll
            for (int nb = 0; nb < C::NB; ++nb)
#pragma unroll
                for (int i = 0; i < 16; ++i) acc[mat][mb][nb][i] = 0.f;

    const int wm = wave / C::WN, wn = wave % C::WN;
    const int l32 = lane & 31, hi8 = (lane >> 5) * 8;
    const int nk = ceil_div(K, BK);

    gemm_gload<C>(ra, rb, p.A, Bm[0], Bm[1], tid, 0, m0, m_end, n0, N, K);
    gemm_sstore<C>(ra, rb, sA, sB, tid, 0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        const bool more = kt + 1 < nk;
        if (more) gemm_gload<C>(ra, rb, p.A, Bm[0], Bm[1], tid, (kt + 1) * BK, m0, m_end, n0, N, K);
        const uint16_t* a_base = sA + (size_t)(buf * BM + wm * C::WTM + l32) * C::LROW + hi8;
#pragma unroll
        for (int kk = 0; kk < BK / 16; ++kk) {
            uint4 af[C::MB];
            uint4 bf[C::NMAT][C::NB];
#pragma unroll
            for (int mb = 0; mb < C::MB; ++mb)
                af[mb] = *(const uint4*)(a_base + mb * 32 * C::LROW + kk * 16);
#pragma unroll
            for (int mat = 0; mat < C::NMAT; ++mat)
#pragma unroll
                for (int nb = 0; nb < C::NB; ++nb)
                    bf[mat][nb] = *(const uint4*)(sB +
                        (size_t)((mat * 2 + buf) * BN + wn * C::WTN + nb * 32 + l32) * C::LROW + hi8 + kk * 16);
#pragma unroll
            for (int mat = 0; mat < C::NMAT; ++mat)
#pragma unroll
                for (int mb = 0; mb < C::MB; ++mb)
#pragma unroll
                    for (int nb = 0; nb < C::NB; ++nb)
                        acc[mat][mb][nb] = mfma32(af[mb], bf[mat][nb], acc[mat][mb][nb]);
        }
        if (more) gemm_sstore<C>(ra, rb, sA, sB, tid, buf ^ 1);
        __syncthreads();
    }

    // ---- epilogue: stage the wave's tile in LDS, then 128-bit row stores
    uint16_t* st = (uint16_t*)smem + (size_t)wave * C::WTM * C::SROW;
#pragma unroll
    for (int mb = 0; mb < C::MB; ++mb)
#pragma unroll
        for (int nb = 0; nb < C::NB; ++nb)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int r = mb * 32 + 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
                const int c = nb * 32 + l32;
                float v;
                if constexpr (GATED) {
                    const float g = acc[0][mb][nb][i], u = acc[1][mb][nb][i];
                    v = g / (1.f + expf(-g)) * u;
                } else {
                    v = acc[0][mb][nb][i];
                }
                st[r * C::SROW + c] = f32_to_bf16(v);
            }
    __syncthreads();
    constexpr int CPR = C::WTN / 8;  // 16-byte chunks per staged row
    const int row0 = m0 + wm * C::WTM, col0 = n0 + wn * C::WTN;
#pragma unroll 4
    for (int c = lane; c < C::WTM * CPR; c += 64) {
        const int r = c / CPR, cc = c % CPR;
        const int gm = row0 + r, gn = col0 + cc * 8;
        if (gm < m_end && gn < N)
            *(uint4*)(p.C + (size_t)gm * N + gn) = *(const uint4*)(st + r * C::SROW + cc * 8);
    }
}

template <bool GATED, int BM, int BN, int BK>
hipError_t launch_gemm(const GemmParams& g, hipStream_t s) {
    const int64_t mt_max = ceil_div64(g.rows_cap, BM) + g.n_seg;
    const int64_t nt = ceil_div64(g.N, BN);
    int64_t blocks = mt_max * nt;
    blocks = (blocks + 7) / 8 * 8;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
    hipLaunchKernelGGL((grouped_gemm_kernel<GATED, BM, BN, BK>), dim3((unsigned)blocks),
                       dim3(kGemmThreads), 0, s, g);
    return hipGetLastError();
}

// ---- f32 path

__device__ __forceinline__ int find_segment(const int32_t* offsets, int n_seg, int rows_cap, int row) {
    for (int q = 0; q < n_seg; ++q) {
        const int b = min(max(offsets[q], 0), rows_cap);
        const int e = min(max(offsets[q + 1], b), rows_cap);
        if (row >= b && row < e) return q;
    }
    return -1;
}

__global__ __launch_bounds__(256) void ffn_f32_gateup_kernel(const float* __restrict__ a,
                                                             const float* __restrict__ wg,
                                                             const float* __restrict__ wu,
                                                             float* __restrict__ h,
                                                             const int32_t* __restrict__ offsets,
                                                             int n_seg, int rows_cap, int d, int d_ff) {
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (idx >= (int64_t)rows_cap * d_ff) return;
    const int row = (int)(idx / d_ff), j = (int)(idx % d_ff);
    const int s = find_segment(offsets, n_seg, rows_cap, row);
    if (s < 0) return;
    const float* ar = a + (size_t)row * d;
    const float* gr = wg + ((size_t)s * d_ff + j) * d;
    const float* ur = wu + ((size_t)s * d_ff + j) * d;
    float g = 0.f, u = 0.f;
    for (int c = 0; c < d; ++c) {
        g = fmaf(ar[c], gr[c], g);
        u = fmaf(ar[c], ur[c], u);
    }
    h[(size_t)row * d_ff + j] = g / (1.f + expf(-g)) * u;
}

__global__ __launch_bounds__(256) void ffn_f32_down_kernel(const float* __restrict__ h,
                                                           const float* __restrict__ wd,
                                                           float* __restrict__ y,
                                                           const int32_t* __restrict__ offsets,
                                                           int n_seg, int rows_cap, int d, int d_ff) {
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (idx >= (int64_t)rows_cap * d) return;
    const int row = (int)(idx / d), i = (int)(idx % d);
    const int s = find_segment(offsets, n_seg, rows_cap, row);
    if (s < 0) return;
    const float* hr = h + (size_t)row * d_ff;
    const float* dr = wd + ((size_t)s * d + i) * d_ff;
    float acc = 0.f;
    for (int j = 0; j < d_ff; ++j) acc = fmaf(hr[j], dr[j], acc);
    y[(size_t)row * d + i] = acc;
}

}  // namespace

hipError_t launch_ffn(const FfnArgs& a, hipStream_t s, int part) {
    if (a.rows_cap == 0) return hipSuccess;
    const bool up = part != 2, down = part != 1;
    if (a.dtype == BMOE_F32) {
        const int64_t n1 = (int64_t)a.rows_cap * a.d_ff, n2 = (int64_t)a.rows_cap * a.d;
        if (up) {
            hipLaunchKernelGGL(ffn_f32_gateup_kernel, dim3((unsigned)ceil_div64(n1, 256)), dim3(256), 0, s,
                               (const float*)a.a, (const float*)a.w_gate, (const float*)a.w_up, (float*)a.h,
                               a.offsets, a.n_seg, a.rows_cap, a.d, a.d_ff);
            hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
        }
        if (down) {
            hipLaunchKernelGGL(ffn_f32_down_kernel, dim3((unsigned)ceil_div64(n2, 256)), dim3(256), 0, s,
                               (const float*)a.h, (const float*)a.w_down, (float*)a.y, a.offsets, a.n_seg,
                               a.rows_cap, a.d, a.d_ff);
            return hipGetLastError();
        }
        return hipSuccess;
    }
    if (up) {
        GemmParams g1{(const uint16_t*)a.a, (const uint16_t*)a.w_gate, (const uint16_t*)a.w_up,
                      (uint16_t*)a.h, a.offsets, a.n_seg, a.rows_cap, a.d_ff, a.d};
        hipError_t e = launch_gemm<true, 128, 128, 64>(g1, s);
        if (e != hipSuccess) return e;
    }
    if (down) {
        GemmParams g2{(const uint16_t*)a.h, (const uint16_t*)a.w_down, nullptr, (uint16_t*)a.y,
                      a.offsets, a.n_seg, a.rows_cap, a.d, a.d_ff};
        return launch_gemm<false, 128, 256, 64>(g2, s);
    }
    return hipSuccess;
}

}  // namespace bmoe
