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
#include <cstdlib>
#include <type_traits>

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
    int sk_min_idle;  // stream-K split threshold (average idle K-steps per workgroup)
    const int32_t* a_rows = nullptr;  // gathered A: row r is A[a_rows[r]] (A has a_count rows)
    int a_count = 0;
    FoldArgs fold;  // combine folded into the down projection's epilogue (out == nullptr: not folded)
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

// arow[i]: source row of this thread's A chunk i (see gemm_arows)
template <class C>
__device__ __forceinline__ void gemm_gload(uint4 (&ra)[C::A_CH], uint4 (&rb)[C::NMAT][C::B_CH],
                                           const uint16_t* A, const int (&arow)[C::A_CH], const uint16_t* B0,
                                           const uint16_t* B1, int tid, int k0, int n0, int N, int K) {
#pragma unroll
    for (int i = 0; i < C::A_CH; ++i) {
        const int c = tid + kGemmThreads * i;
        const int cc = c % C::KCH;
        const int gk = k0 + cc * 8;
        ra[i] = gk < K ? *(const uint4*)(A + (size_t)arow[i] * K + gk) : make_uint4(0, 0, 0, 0);
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

// source rows of this thread's A chunks for the tile's rows [m0, m_end)
// (clamped to the last row; gathered through a_rows when the operand is)
template <class C>
__device__ __forceinline__ void gemm_arows(int (&arow)[C::A_CH], const GemmParams& p, int tid, int m0, int m_end) {
#pragma unroll
    for (int i = 0; i < C::A_CH; ++i) {
        const int c = tid + kGemmThreads * i;
        arow[i] = gathered_row(p.a_rows, p.a_count, min(m0 + c / C::KCH, m_end - 1));
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

template <class C>
__device__ __forceinline__ void gemm_frags(uint4 (&af)[C::MB], uint4 (&bf)[C::NMAT][C::NB],
                                           const uint16_t* a_base, const uint16_t* b_base, int kk) {
    constexpr int BN = C::B_CH * kGemmThreads / C::KCH;
#pragma unroll
    for (int mb = 0; mb < C::MB; ++mb) af[mb] = *(const uint4*)(a_base + mb * 32 * C::LROW + kk * 16);
#pragma unroll
    for (int mat = 0; mat < C::NMAT; ++mat)
#pragma unroll
        for (int nb = 0; nb < C::NB; ++nb)
            bf[mat][nb] = *(const uint4*)(b_base + (size_t)(mat * 2 * BN + nb * 32) * C::LROW + kk * 16);
}

template <class C>
__device__ __forceinline__ void gemm_mfmas(f32x16 (&acc)[C::NMAT][C::MB][C::NB], const uint4 (&af)[C::MB],
                                           const uint4 (&bf)[C::NMAT][C::NB]) {
#pragma unroll
    for (int mat = 0; mat < C::NMAT; ++mat)
#pragma unroll
        for (int mb = 0; mb < C::MB; ++mb)
#pragma unroll
            for (int nb = 0; nb < C::NB; ++nb) acc[mat][mb][nb] = mfma32(af[mb], bf[mat][nb], acc[mat][mb][nb]);
}

template <bool GATED, int BM, int BN, int BK, bool FDB>
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

    int arow[C::A_CH];
    gemm_arows<C>(arow, p, tid, m0, m_end);
    gemm_gload<C>(ra, rb, p.A, arow, Bm[0], Bm[1], tid, 0, n0, N, K);
    gemm_sstore<C>(ra, rb, sA, sB, tid, 0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        const bool more = kt + 1 < nk;
        if (more) gemm_gload<C>(ra, rb, p.A, arow, Bm[0], Bm[1], tid, (kt + 1) * BK, n0, N, K);
        const uint16_t* a_base = sA + (size_t)(buf * BM + wm * C::WTM + l32) * C::LROW + hi8;
        const uint16_t* b_base = sB + (size_t)(buf * BN + wn * C::WTN + l32) * C::LROW + hi8;
        if constexpr (FDB) {
            // fragments of sub-step kk+1 are read from LDS while sub-step kk runs on the MFMA pipe
            uint4 af[2][C::MB];
            uint4 bf[2][C::NMAT][C::NB];
            gemm_frags<C>(af[0], bf[0], a_base, b_base, 0);
#pragma unroll
            for (int kk = 0; kk < BK / 16; ++kk) {
                const int cur = kk & 1;
                if (kk + 1 < BK / 16) gemm_frags<C>(af[cur ^ 1], bf[cur ^ 1], a_base, b_base, kk + 1);
                gemm_mfmas<C>(acc, af[cur], bf[cur]);
            }
        } else {
#pragma unroll
            for (int kk = 0; kk < BK / 16; ++kk) {
                uint4 af[C::MB];
                uint4 bf[C::NMAT][C::NB];
                gemm_frags<C>(af, bf, a_base, b_base, kk);
                gemm_mfmas<C>(acc, af, bf);
            }
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

template <bool GATED, int BM, int BN, int BK, bool FDB>
hipError_t launch_gemm(const GemmParams& g, hipStream_t s) {
    const int64_t mt_max = ceil_div64(g.rows_cap, BM) + g.n_seg;
    const int64_t nt = ceil_div64(g.N, BN);
    int64_t blocks = mt_max * nt;
    blocks = (blocks + 7) / 8 * 8;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
    hipLaunchKernelGGL((grouped_gemm_kernel<GATED, BM, BN, BK, FDB>), dim3((unsigned)blocks),
                       dim3(kGemmThreads), 0, s, g);
    return hipGetLastError();
}

// ---- bf16 grouped GEMM with direct global->LDS loads (K % BK == 0)
//
// 256 x 256 workgroup tile (gate/up: 128 columns of each matrix), 128 x 128
// per wave, a ring of LDS stages filled by global_load_lds_dwordx4 (no
// staging registers, no LDS store instructions). A stage holds every tile
// row's BK k-values as one LDS row of BK*2 bytes whose 16-byte chunks are
// XOR-swizzled by (row >> 1), so the 32 rows of an MFMA fragment read without
// bank conflicts; one DMA instruction fills 64/(BK/8) consecutive rows, each
// lane fetching the global chunk that belongs in its LDS slot (the lanes of a
// row read the row's contiguous bytes). The DMA and the barrier are issued
// through inline asm: with the builtin, the compiler would wait for every
// outstanding DMA before each LDS read and at each barrier, defeating the ring.
// Per K-step (four MFMA sub-steps of k = 16): by the end of sub-step 0
// every fragment of the stage is in registers (sub-steps 0 and 1 were read
// during the previous K-step), and a barrier releases its slot; sub-steps
// 1-3 issue the copies of K-step kt+2 into it (6, 5 and 5 per wave); after
// sub-step 2 a wait for this wave's older copies and a second barrier make
// K-step kt+1 resident, and sub-step 3 reads its first two sub-steps.

// K-step and ring depth of the DMA kernels. BK = 64 makes every DMA row a
// full 128-byte line (8 rows per instruction), which the L2 and MALL serve
// faster than 64-byte pieces; two 64 KB stages leave one stage in flight.
// Measured on the grouped workloads, more stages of BK = 32 did not help:
// the pipeline is bound by L2/MALL throughput, not by latency.
// ---- bf16 grouped GEMM with direct-to-LDS copies (large groups)
//
// 256x256 workgroup tile (gate/up: 128 columns of each of W_gate and W_up, so
// SiLU(gate)*up happens in the epilogue), 128x128 per wave, 32x32x16 bf16 MFMA
// with fp32 accumulators, K-step 64 through a two-slot LDS ring filled by
// global_load_lds_dwordx4.
//
// Work distribution. Without a workspace every workgroup computes one tile.
// With one (stream-K), the grid is one workgroup per CU: full rounds of one
// tile per workgroup, then the K-steps of the remaining tiles (between one
// and two rounds' worth) are split evenly across the workgroups. A workgroup
// whose share starts or ends inside a tile writes that piece's fp32
// accumulators to its workspace slot, and a second kernel sums the pieces of
// each split tile in K order and applies the epilogue. No workgroup ever
// waits for another, so nothing depends on which workgroups are resident.

constexpr int kGroupM = 8;
constexpr int kDmaBK = 64;
constexpr int kSkPartBytes = 256 * 256 * 4;  // fp32 accumulators of one tile piece
// workspace slot stride: a piece plus 1280 bytes, so that slots (which the
// workgroups write, and the fixup reads, at the same offsets at the same
// time) do not all start on the same memory channel
constexpr int kSkSlotBytes = kSkPartBytes + 1280;

template <bool GATED>
struct DmaCfg {
    static constexpr int BM = 256, BK = kDmaBK, KC = BK / 8;  // KC: 16-byte chunks per row
    static constexpr int SUB = BK / 16;                       // MFMA sub-steps per K-step
    static constexpr int BN = GATED ? 128 : 256;              // output columns per matrix
    static constexpr int NMAT = GATED ? 2 : 1;
    static constexpr int RB = NMAT * BN;                      // B rows staged per K-step (256)
    static constexpr int WTM = BM / 2, WTN = BN / 2;
    static constexpr int MB = WTM / 32, NB = WTN / 32;
    static constexpr int ROW_BYTES = BK * 2;
    static constexpr int ROWS_PER_DMA = 64 / KC;              // rows one DMA instruction fills
    static constexpr int A_DMA = BM / (4 * ROWS_PER_DMA);     // per wave per K-step
    static constexpr int B_DMA = RB / (4 * ROWS_PER_DMA);
    static constexpr int DMA_PER_STAGE = A_DMA + B_DMA;
    static constexpr int A_STAGE = BM * ROW_BYTES, B_STAGE = RB * ROW_BYTES;
    static constexpr int STAGE = A_STAGE + B_STAGE;
    static constexpr int SROW = WTN + 8;
    static constexpr int RING = 2 * STAGE;
    // epilogue staging: each wave its own 16 rows x WTN, outside the ring, so
    // the next tile's first copies can land while a tile's results go out
    static constexpr int HSTG = 16 * SROW * 2;
    static constexpr int STG_OFF = RING;
    static constexpr int SCHED_OFF = STG_OFF + 4 * HSTG;                 // schedule arrays after them
    static constexpr int SCHED = (256 + 3 * BMOE_MAX_EXPERTS + 1) * 4;
    static constexpr int SMEM = SCHED_OFF + SCHED;
    static constexpr int CPR = WTN / 8;                                   // 16-byte chunks per output row
    static constexpr int NACC4 = NMAT * MB * NB * 4;                      // float4 accumulators per lane
    static_assert(KC == 8 && BM == 256 && RB == 256, "tile shape");
    static_assert(SUB % 2 == 0, "fragment double buffer alternates within a K-step");
    static_assert(SMEM <= 160 * 1024, "LDS of one workgroup");
    static_assert(NACC4 * 16 * kGemmThreads == kSkPartBytes, "piece size");
};

// 16-byte chunk swizzle of a tile row: conflict-free 128-bit fragment reads
template <int KC>
__device__ __forceinline__ int swz(int row) { return (row >> 1) & (KC - 1); }

// LDS byte offset of logical 16-byte chunk c of tile row r within a stage region
template <class C>
__device__ __forceinline__ int lds_off(int r, int c) { return r * C::ROW_BYTES + ((c ^ swz<C::KC>(r)) << 4); }

// Zero-filled rows (device memory of the library, zero at load time): the
// copies of A rows wholly past a segment's end read these instead of the
// segment's last row, so the MFMAs of padding rows see zero operands.
constexpr int kZeroBytes = 64 * 1024 + 128;
__device__ __align__(256) uint16_t g_zero_rows[kZeroBytes / 2];

// Copy sources of one wave: a workgroup-uniform base per operand (SGPRs) and
// a 32-bit byte offset per lane and instruction (one VGPR each). Bit i of
// a_zero: A instruction i's rows all lie past the segment's end (it copies
// from g_zero_rows).
template <class C>
struct DmaSrc {
    const char* a_base;
    const char* b_base;
    uint32_t a_off[C::A_DMA];
    uint32_t b_off[C::B_DMA];
    int a_zero;
};

// DMA instruction i of the wave's share of a K-step: instructions 0..A_DMA-1
// fill A rows, the rest B rows; instruction i of wave w fills ROWS_PER_DMA
// consecutive rows (1 KB of LDS). kb: byte offset of the K-step in a row.
template <class C>
__device__ __forceinline__ void dma_one(const DmaSrc<C>& src, uint32_t stage_lds, int wave, int kb, int i) {
    if (i < C::A_DMA) {
        const char* base = (src.a_zero >> i) & 1 ? (const char*)g_zero_rows : src.a_base;
        dma16s(base + kb, src.a_off[i], stage_lds + ((wave * C::A_DMA + i) * C::ROWS_PER_DMA) * C::ROW_BYTES);
    } else {
        const int j = i - C::A_DMA;
        dma16s(src.b_base + kb, src.b_off[j],
               stage_lds + C::A_STAGE + ((wave * C::B_DMA + j) * C::ROWS_PER_DMA) * C::ROW_BYTES);
    }
}

template <class C>
__device__ __forceinline__ void dma_stage(const DmaSrc<C>& src, uint32_t stage_lds, int wave, int kb) {
#pragma unroll
    for (int i = 0; i < C::DMA_PER_STAGE; ++i) dma_one<C>(src, stage_lds, wave, kb, i);
}

// First tile row of 32-row block mb of wave row wm. (Interleaving the two
// wave rows' blocks and leaving out the MFMAs of blocks wholly past a
// segment's end made the partly filled last tiles of the segments run ahead
// of the others: the workgroups of an XCD then drifted apart along K, and the
// gate/up GEMM's L2 misses doubled. Every tile keeps the full MFMA work.)
template <class C>
__device__ __forceinline__ int dma_arow(int wm, int mb) { return wm * C::WTM + mb * 32; }

template <class C>
__device__ __forceinline__ void dma_frags(uint4 (&af)[C::MB], uint4 (&bf)[C::NMAT][C::NB], const char* stage,
                                          int wm, int wn, int lane, int kk) {
    const int c = kk * 2 + (lane >> 5), l32 = lane & 31;
#pragma unroll
    for (int mb = 0; mb < C::MB; ++mb)
        af[mb] = *(const uint4*)(stage + lds_off<C>(dma_arow<C>(wm, mb) + l32, c));
#pragma unroll
    for (int mat = 0; mat < C::NMAT; ++mat)
#pragma unroll
        for (int nb = 0; nb < C::NB; ++nb)
            bf[mat][nb] = *(const uint4*)(stage + C::A_STAGE + lds_off<C>(mat * C::BN + wn * C::WTN + nb * 32 + l32, c));
}

// Fragment read r of a sub-step (r < NMAT*NB: B fragments, then A).
template <class C>
__device__ __forceinline__ void frag_read(uint4 (&ga)[C::MB], uint4 (&gb)[C::NMAT][C::NB], const char* stage, int wm,
                                          int wn, int l32, int c, int r) {
    if (r < C::NMAT * C::NB) {
        const int rm = r / C::NB, rn = r % C::NB;
        gb[rm][rn] = *(const uint4*)(stage + C::A_STAGE + lds_off<C>(rm * C::BN + wn * C::WTN + rn * 32 + l32, c));
    } else {
        const int ra = r - C::NMAT * C::NB;
        ga[ra] = *(const uint4*)(stage + lds_off<C>(dma_arow<C>(wm, ra) + l32, c));
    }
}

// The MFMAs of one sub-step with, between them, the fragment reads of RD
// later sub-steps (RD = 1: one read after every second MFMA; RD = 2: one
// after every MFMA, set 1 first) and ND of the wave's copies of a K-step
// (DMA instructions d0 .. d0 + ND - 1), one after every (NM / ND)-th MFMA.
// (Issuing a sub-step's copies after each of its first MFMAs instead
// measured 1-3 % slower: the copies must be spread.)
template <class C, int RD, int ND>
__device__ __forceinline__ void mfmas_ops(f32x16 (&acc)[C::NMAT][C::MB][C::NB], const uint4 (&af)[C::MB],
                                          const uint4 (&bf)[C::NMAT][C::NB], uint4 (&ga1)[C::MB],
                                          uint4 (&gb1)[C::NMAT][C::NB], const char* st1, int kk1,
                                          uint4 (&ga2)[C::MB], uint4 (&gb2)[C::NMAT][C::NB], const char* st2,
                                          int kk2, int wm, int wn, int lane, const DmaSrc<C>& src,
                                          uint32_t dma_lds, int wave, int kb, int d0) {
    constexpr int NM = C::NMAT * C::MB * C::NB, NR = C::MB + C::NMAT * C::NB;
    static_assert(2 * NR == NM && C::DMA_PER_STAGE == NM, "one read and one copy per two MFMAs");
    static_assert(ND >= 0 && ND <= NM / 2, "at most one copy per two MFMAs");
    constexpr int STEP = ND > 0 ? NM / ND : NM;
    const int l32 = lane & 31, c1 = kk1 * 2 + (lane >> 5), c2 = kk2 * 2 + (lane >> 5);
#pragma unroll
    for (int q = 0; q < NM; ++q) {
        const int mb = q / (C::NMAT * C::NB), mat = (q / C::NB) % C::NMAT, nb = q % C::NB;
        acc[mat][mb][nb] = mfma32(af[mb], bf[mat][nb], acc[mat][mb][nb]);
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (RD == 2) {
            if (q < NR) frag_read<C>(ga1, gb1, st1, wm, wn, l32, c1, q);
            else frag_read<C>(ga2, gb2, st2, wm, wn, l32, c2, q - NR);
        } else if constexpr (RD == 1) {
            if (q & 1) frag_read<C>(ga1, gb1, st1, wm, wn, l32, c1, q >> 1);
        }
        if constexpr (ND > 0) {
            if (q % STEP == 0 && q / STEP < ND) dma_one<C>(src, dma_lds, wave, kb, d0 + q / STEP);
        }
        __builtin_amdgcn_sched_barrier(0);
    }
}

// ---- tile schedule: per-segment M-tile prefix in LDS, computed from the
// device offsets by every workgroup (the host does not read the offsets)
struct TileSched {
    int* s_mt;   // [n_seg + 1] first M-tile of each segment
    int* s_beg;  // [n_seg] first row of each segment
    int* s_end;  // [n_seg] end row of each segment
    int NT, total_mt;
};

struct TileCoord {
    int s, m0, m_end, n0;
};

// Returns the schedule; ends with a barrier. The arrays must not be written
// while a workgroup uses them (they live outside the ring and staging area).
__device__ __forceinline__ TileSched tile_sched(const GemmParams& p, char* sched_lds, int BM, int BN) {
    TileSched t;
    int* s_scan = (int*)sched_lds;
    t.s_mt = s_scan + 256;
    t.s_beg = t.s_mt + BMOE_MAX_EXPERTS + 1;
    t.s_end = t.s_beg + BMOE_MAX_EXPERTS;
    const int tid = threadIdx.x;
    int cnt = 0;
    if (tid < p.n_seg) {
        const int beg = min(max(p.offsets[tid], 0), p.rows_cap);
        const int end = min(max(p.offsets[tid + 1], beg), p.rows_cap);
        t.s_beg[tid] = beg;
        t.s_end[tid] = end;
        cnt = ceil_div(end - beg, BM);
    }
    int total_mt;
    const int ex = block_exclusive_scan_256(cnt, s_scan, &total_mt);
    if (tid < p.n_seg) t.s_mt[tid] = ex;
    if (tid == 0) t.s_mt[p.n_seg] = total_mt;
    __syncthreads();
    t.total_mt = __builtin_amdgcn_readfirstlane(total_mt);
    t.NT = ceil_div(p.N, BN);
    return t;
}

// Tile L of the schedule: segments in order; inside a segment, groups of
// kGroupM M-tiles with N-tiles outer, so that the workgroups that run
// together on one XCD share A and B panels in L2. The values come from LDS;
// readfirstlane keeps them (and the copy bases) in SGPRs.
__device__ __forceinline__ TileCoord tile_coord(const TileSched& t, int n_seg, int L, int BM, int BN) {
    const int NT = t.NT;
    int lo = 0, hi = n_seg - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (t.s_mt[mid] * NT <= L) lo = mid;
        else hi = mid - 1;
    }
    TileCoord c;
    c.s = __builtin_amdgcn_readfirstlane(lo);
    const int mts = __builtin_amdgcn_readfirstlane(t.s_mt[c.s + 1] - t.s_mt[c.s]);
    const int local = L - __builtin_amdgcn_readfirstlane(t.s_mt[c.s]) * NT;
    const int mg = local / (kGroupM * NT), gm = min(kGroupM, mts - mg * kGroupM);
    const int rem = local - mg * kGroupM * NT;
    const int nt = rem / gm, mt = mg * kGroupM + rem % gm;
    c.m0 = __builtin_amdgcn_readfirstlane(t.s_beg[c.s]) + mt * BM;
    c.m_end = __builtin_amdgcn_readfirstlane(t.s_end[c.s]);
    c.n0 = nt * BN;
    return c;
}

template <class C, bool GATED>
__device__ __forceinline__ void dma_sources(DmaSrc<C>& src, const GemmParams& p, const TileCoord& tc, int wave,
                                            int lane_in) {
    const int K = p.K, N = p.N;
    // the lane-dependent parts are recomputed for every tile (a few integer
    // operations): held across the persistent loop they were spilled to
    // scratch and reloaded one dependent load at a time
    int lane = lane_in;
    asm volatile("" : "+v"(lane));
    const int lrow = lane / C::KC, lchk = lane % C::KC;
    // offsets from the tile's first row, or from row 0 of the source when the
    // rows are gathered (the host keeps a_count * K * 2 below 2^32)
    const int base_row = p.a_rows ? 0 : tc.m0;
    src.a_base = (const char*)(p.A + (size_t)base_row * K);
    // an instruction whose rows all lie past the segment's end copies zeros
    // (row stride 0 into g_zero_rows, which holds a whole row of K columns)
    const bool zero_ok = (size_t)K * 2 + 128 <= (size_t)kZeroBytes;
    int a_zero = 0;
#pragma unroll
    for (int i = 0; i < C::A_DMA; ++i) {
        const int r = (wave * C::A_DMA + i) * C::ROWS_PER_DMA + lrow;
        const bool z = zero_ok && tc.m0 + (wave * C::A_DMA + i) * C::ROWS_PER_DMA >= tc.m_end;
        a_zero |= z ? 1 << i : 0;
        const int row = gathered_row(p.a_rows, p.a_count, min(tc.m0 + r, tc.m_end - 1));
        src.a_off[i] = z ? (uint32_t)(lchk << 4)
                         : (uint32_t)(((size_t)(row - base_row) * K + ((lchk ^ swz<C::KC>(r)) << 3)) * 2);
    }
    src.a_zero = __builtin_amdgcn_readfirstlane(a_zero);
    // a wave's B rows lie in one matrix (gate or up for the gated GEMM)
    static_assert(!GATED || (C::B_DMA * C::ROWS_PER_DMA * 2 == C::BN), "B rows of a wave in one matrix");
    const int bmat = GATED ? (wave * C::B_DMA * C::ROWS_PER_DMA) / C::BN : 0;
    src.b_base = (const char*)((bmat ? p.B1 : p.B0) + ((size_t)tc.s * N + tc.n0) * K);
#pragma unroll
    for (int i = 0; i < C::B_DMA; ++i) {
        const int r = (wave * C::B_DMA + i) * C::ROWS_PER_DMA + lrow;
        const int n = min(tc.n0 + r % C::BN, N - 1);
        src.b_off[i] = (uint32_t)(((n - tc.n0) * K + ((lchk ^ swz<C::KC>(r)) << 3)) * 2);
    }
}

// The copies of K-steps ka and ka+1 (when the item has two) into the ring's
// two slots; the ring must be free (every wave done reading it).
template <class C>
__device__ __forceinline__ void ksteps_prologue(const DmaSrc<C>& src, char* smem, int ka, int kb, int wave) {
    const uint32_t lds0 = (uint32_t)(uintptr_t)smem;
    dma_stage<C>(src, lds0, wave, ka * C::BK * 2);
    if (kb - ka > 1) dma_stage<C>(src, lds0 + C::STAGE, wave, (ka + 1) * C::BK * 2);
}

// What a wave issued to vector memory after its prologue copies: nothing, or
// the previous item's epilogue stores. The first wait then counts only the
// second K-step's copies, or waits for everything (stores included: the
// counter is not relied on to order the copies before later stores).
enum { kAfterNone = 0, kAfterStores = 1 };

// K-steps [ka, kb) of one tile into acc (which the caller zeroed), after
// their first two K-steps' copies were issued (ksteps_prologue, or the
// previous item's last K-steps). K-step kt lives in ring slot (kt + s0) & 1.
// The next item (tile tc2, K-steps [nka, nkb); nka == nkb: none) has its
// first two K-steps copied as if they continued this item's: once this
// item's own copies are all issued, src is set to the next item's sources
// and its K-steps nka and nka+1 go into the slots this item's last two
// K-steps free, so they arrive while this item's results go out (an item of
// one K-step copies the next item's first K-step after its loop). Ends with
// a barrier; src then holds the next item's sources.
template <class C, bool GATED>
__device__ __forceinline__ void tile_ksteps(f32x16 (&acc)[C::NMAT][C::MB][C::NB], DmaSrc<C>& src, char* smem,
                                            int ka, int kb, int wave, int lane, int after, int s0,
                                            const GemmParams& p, const TileCoord& tc2, int nka, int nkb) {
    const uint32_t lds0 = (uint32_t)(uintptr_t)smem;
    const int wm = wave >> 1, wn = wave & 1;
    const int n = kb - ka, nn = nkb - nka;
    // wait for K-step ka: vector-memory operations complete in issue order, so
    // at most (its successors) may still be outstanding
    if (after == kAfterNone && n > 1) wait_vmcnt<C::DMA_PER_STAGE>();
    else wait_vmcnt<0>();
    wg_barrier();
    // Fragments two sub-steps ahead, in four register sets (set j holds
    // sub-step j of a K-step). Sub-step j reads sub-step j+2 (the next
    // K-step's slot for j >= 2). After sub-step 1 every fragment of this
    // K-step's slot is in registers: one barrier then releases the slot and
    // (after this wave's wait) makes the next K-step's slot resident, and
    // sub-steps 2 and 3 issue the copies of K-step kt+2 into the released
    // slot, one per two MFMAs.
    static_assert(C::SUB == 4, "four sub-steps per K-step");
    uint4 af[4][C::MB];
    uint4 bf[4][C::NMAT][C::NB];
    // Sub-step 0 reads sub-steps 2 and 3, so a barrier after it releases the
    // slot; sub-steps 1-3 issue the copies of K-step kt+2 (6, 5, 5); after
    // sub-step 2 a wait for this wave's older copies and a second barrier
    // make K-step kt+1 resident; sub-step 3 reads its sub-steps 0 and 1.
    dma_frags<C>(af[0], bf[0], smem + (s0 & 1) * C::STAGE, wm, wn, lane, 0);
    dma_frags<C>(af[1], bf[1], smem + (s0 & 1) * C::STAGE, wm, wn, lane, 1);
    // K-step kt; with DMA, the copies of K-step kbyte / (BK * 2) of src go
    // into its slot once the slot is free
    auto kstep = [&](int kt, auto with_dma, int kbyte) {
        const DmaSrc<C>& cs = src;
        constexpr bool DMA = decltype(with_dma)::value;
        const int slot = (kt + s0) & 1;
        const char* cur = smem + slot * C::STAGE;
        const char* nxt = smem + (slot ^ 1) * C::STAGE;
        const uint32_t dma_lds = lds0 + slot * C::STAGE;
        const int kb = kbyte;
        constexpr int D1 = 6, D2 = 5, D3 = C::DMA_PER_STAGE - D1 - D2;
        __builtin_amdgcn_sched_barrier(0);
        mfmas_ops<C, 2, 0>(acc, af[0], bf[0], af[2], bf[2], cur, 2, af[3], bf[3], cur, 3, wm, wn, lane, cs,
                           dma_lds, wave, kb, 0);
        __builtin_amdgcn_sched_barrier(0);
        lds_reads_done();
        wg_barrier();  // the slot is free
        __builtin_amdgcn_sched_barrier(0);
        mfmas_ops<C, 0, DMA ? D1 : 0>(acc, af[1], bf[1], af[1], bf[1], cur, 0, af[1], bf[1], cur, 0, wm, wn, lane,
                                      cs, dma_lds, wave, kb, 0);
        __builtin_amdgcn_sched_barrier(0);
        mfmas_ops<C, 0, DMA ? D2 : 0>(acc, af[2], bf[2], af[2], bf[2], cur, 0, af[2], bf[2], cur, 0, wm, wn, lane,
                                      cs, dma_lds, wave, kb, D1);
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (DMA) wait_vmcnt<D1 + D2>();
        else wait_vmcnt<0>();
        wg_barrier();  // the next K-step is resident
        __builtin_amdgcn_sched_barrier(0);
        mfmas_ops<C, 2, DMA ? D3 : 0>(acc, af[3], bf[3], af[0], bf[0], nxt, 0, af[1], bf[1], nxt, 1, wm, wn, lane,
                                      cs, dma_lds, wave, kb, D1 + D2);
        __builtin_amdgcn_sched_barrier(0);
    };
    int kt = 0;
    for (; kt + 2 < n; ++kt) kstep(kt, std::true_type{}, (ka + kt + 2) * C::BK * 2);
    // this item's copies are all issued: the last two K-steps copy K-steps
    // j = kt + 2 - n of the next item; where it has no such K-step (or there
    // is no next item) they copy one it (or this item) has into the free
    // slot, which nothing reads (one code path, no branch between K-steps)
    if (nn > 0) dma_sources<C, GATED>(src, p, tc2, wave, lane);
    for (; kt < n; ++kt) {
        const int j = kt + 2 - n;
        const int kj = nn > 0 ? nka + min(j, nn - 1) : ka;
        kstep(kt, std::true_type{}, kj * C::BK * 2);
    }
    // no next item: the last copies (into free slots) complete before the
    // workgroup can end, so none lands in a later workgroup's LDS
    if (nn == 0) wait_vmcnt<0>();
    __syncthreads();
    // an item of one K-step issued only the next item's second K-step: its
    // first goes in now (the ring is free after the barrier)
    if (n == 1 && nn > 0) dma_stage<C>(src, lds0 + ((n + s0) & 1) * C::STAGE, wave, nka * C::BK * 2);
}

template <class C>
__device__ __forceinline__ void zero_acc(f32x16 (&acc)[C::NMAT][C::MB][C::NB]) {
#pragma unroll
    for (int mat = 0; mat < C::NMAT; ++mat)
#pragma unroll
        for (int mb = 0; mb < C::MB; ++mb)
#pragma unroll
            for (int nb = 0; nb < C::NB; ++nb)
#pragma unroll
                for (int i = 0; i < 16; ++i) acc[mat][mb][nb][i] = 0.f;
}

// An accumulator moved out of its AGPR at the point of use (the compiler
// otherwise copies every accumulator to VGPRs at once after the K loop and,
// inside the persistent loop, spills to scratch).
__device__ __forceinline__ float acc_read(float a) {
    float v;
    asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(v) : "a"(a));
    return v;
}

// Epilogue: the wave's tile (SiLU(gate)*up for the gated GEMM) goes out 16
// rows at a time: staged as bf16 in the wave's own LDS area (outside the
// copy ring), read back in 16-byte row chunks and stored with 128-bit
// stores, with no workgroup barrier.
// With a piece slot instead, the raw fp32 accumulators go to the slot
// (lane-interleaved float4, the layout the fixup reads). One routine for
// both, block by block: with two routines the compiler moved every
// accumulator out of the AGPRs where the paths split and spilled.
// ---- combine folded into the down projection's epilogue
//
// y is still written (as the unfused path writes it), with stores that are
// coherent across the XCDs' L2 caches (sc1: written through to the device's
// coherence point). Once a wave's stores of its 128 columns are complete, it
// counts each of its rows in a counter per (token, 128-column chunk); the row
// that brings a counter to the token's number of rows completes that chunk of
// the token, and its wave forms the chunk of out exactly as the combine kernel
// would: fp32 fmaf of slot gate and bf16 y over the token's valid slots in
// slot order (+ the shared-expert output), one RNE rounding. The other rows
// of the token are read with coherent (sc1) loads; the counter is left zero.
// Whatever order the rows arrive in, out is bit-identical to the unfused
// combine.
typedef uint32_t fold_u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void store_coherent(uint16_t* p, const uint4& v) {
    const fold_u32x4 w = __builtin_bit_cast(fold_u32x4, v);
    asm volatile("global_store_dwordx4 %0, %1, off sc1" ::"v"(p), "v"(w) : "memory");
}
__device__ __forceinline__ uint4 load_coherent(const uint16_t* p) {
    fold_u32x4 w;
    asm volatile("global_load_dwordx4 %0, %1, off sc1\n\ts_waitcnt vmcnt(0)" : "=v"(w) : "v"(p) : "memory");
    return __builtin_bit_cast(uint4, w);
}

// The wave's 128 rows of one tile, columns [c0, c0 + 128) of y, are written
// (and complete): count them, and finish the token chunks they complete.
template <class C>
__device__ __forceinline__ void fold_rows(const GemmParams& p, const TileCoord& tc, int wm, int c0, int lane) {
    const FoldArgs& f = p.fold;
    if (c0 >= p.N) return;  // the wave's columns lie past the row end
    const int k = f.k, chunk = c0 / 128, nchunk = p.N / 128;
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
        const int lr = hh * 64 + lane;  // the wave's local row
        const int gm = tc.m0 + dma_arow<C>(wm, lr / 32) + lr % 32;
        bool last = false;
        int t = 0;
        if (gm < tc.m_end) {
            t = f.perm_token[gm];
            int nrow = 0;
            for (int i = 0; i < k; ++i) nrow += f.slot_row[(size_t)t * k + i] >= 0 ? 1 : 0;
            const int old = __hip_atomic_fetch_add(f.cnt + (size_t)t * nchunk + chunk, 1, __ATOMIC_RELAXED,
                                                   __HIP_MEMORY_SCOPE_AGENT);
            last = old == nrow - 1;
        }
        // the completed chunks, four at a time (16 lanes of 8 columns each)
        uint64_t m = __ballot(last);
        while (m != 0ull) {
            // lane group grp takes the grp-th lowest completing row (if any)
            const int grp = lane >> 4, j = lane & 15;
            uint64_t mm = m;
            for (int q = 0; q < grp; ++q) mm &= mm - 1ull;
            const int src = mm != 0ull ? __ffsll((unsigned long long)mm) - 1 : -1;
            for (int q = 0; q < 4; ++q) m &= m - 1ull;  // (m &= m - 1 is a no-op once m is 0)
            const int tt = __shfl(t, src < 0 ? 0 : src);
            if (src < 0) continue;
            const int col = c0 + j * 8;
            float acc[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[e] = 0.f;
            for (int i = 0; i < k; ++i) {
                const int r = f.slot_row[(size_t)tt * k + i];
                if (r < 0) continue;
                const float g = f.slot_gate[(size_t)tt * k + i];
                const uint4 v = load_coherent(p.C + (size_t)r * p.N + col);
                const uint32_t* u = (const uint32_t*)&v;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    acc[2 * e] = fmaf(g, __uint_as_float(u[e] << 16), acc[2 * e]);
                    acc[2 * e + 1] = fmaf(g, __uint_as_float(u[e] & 0xffff0000u), acc[2 * e + 1]);
                }
            }
            if (f.y_shared) {
                const uint4 v = *(const uint4*)(f.y_shared + (size_t)tt * p.N + col);
                const uint32_t* u = (const uint32_t*)&v;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    acc[2 * e] += __uint_as_float(u[e] << 16);
                    acc[2 * e + 1] += __uint_as_float(u[e] & 0xffff0000u);
                }
            }
            uint4 o;
            o.x = pack_bf16x2(acc[0], acc[1]);
            o.y = pack_bf16x2(acc[2], acc[3]);
            o.z = pack_bf16x2(acc[4], acc[5]);
            o.w = pack_bf16x2(acc[6], acc[7]);
            *(uint4*)(f.out + (size_t)tt * p.N + col) = o;
            if (j == 0)
                __hip_atomic_store(f.cnt + (size_t)tt * nchunk + chunk, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

template <class C, bool GATED, bool FOLD = false>
__device__ __forceinline__ void store_tile(const f32x16 (&acc)[C::NMAT][C::MB][C::NB], const GemmParams& p,
                                           const TileCoord& tc, char* smem, int wave, int lane,
                                           char* piece = nullptr) {
    const int wm = wave >> 1, wn = wave & 1;
    uint16_t* st = (uint16_t*)(smem + C::STG_OFF + wave * C::HSTG);
    const int l32 = lane & 31;
    const int row0 = tc.m0, col0 = tc.n0 + wn * C::WTN;
    if (piece) {
        float4* d = (float4*)piece;
#pragma unroll
        for (int mb = 0; mb < C::MB; ++mb)
#pragma unroll
            for (int nb = 0; nb < C::NB; ++nb) {
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int mat = 0; mat < C::NMAT; ++mat)
#pragma unroll
                    for (int i = 0; i < 16; i += 4) {
                        const int q = ((mat * C::MB + mb) * C::NB + nb) * 4 + i / 4;
                        d[q * kGemmThreads + threadIdx.x] =
                            make_float4(acc_read(acc[mat][mb][nb][i]), acc_read(acc[mat][mb][nb][i + 1]),
                                        acc_read(acc[mat][mb][nb][i + 2]),
                                        acc_read(acc[mat][mb][nb][i + 3]));
                    }
            }
        return;
    }
#pragma unroll
    for (int mb = 0; mb < C::MB; ++mb) {
        if (row0 + dma_arow<C>(wm, mb) >= tc.m_end) continue;  // a block wholly past the segment
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            // rows 16h .. 16h+15 of the 32-row block: accumulator elements 8h .. 8h+7
            __builtin_amdgcn_sched_barrier(0);
            // the half block's values first, each step over all of them, so
            // the SiLU chains (exp, add, reciprocal, products) of different
            // elements overlap instead of running one after another
            float v[C::NB][8];
#pragma unroll
            for (int nb = 0; nb < C::NB; ++nb)
#pragma unroll
                for (int e = 0; e < 8; ++e) v[nb][e] = acc_read(acc[0][mb][nb][8 * h + e]);
            if constexpr (GATED) {
                float u[C::NB][8], t[C::NB][8];
#pragma unroll
                for (int nb = 0; nb < C::NB; ++nb)
#pragma unroll
                    for (int e = 0; e < 8; ++e) u[nb][e] = acc_read(acc[1][mb][nb][8 * h + e]);
#pragma unroll
                for (int nb = 0; nb < C::NB; ++nb)
#pragma unroll
                    for (int e = 0; e < 8; ++e) t[nb][e] = __expf(-v[nb][e]);
#pragma unroll
                for (int nb = 0; nb < C::NB; ++nb)
#pragma unroll
                    for (int e = 0; e < 8; ++e) t[nb][e] = __builtin_amdgcn_rcpf(1.f + t[nb][e]);
#pragma unroll
                for (int nb = 0; nb < C::NB; ++nb)
#pragma unroll
                    for (int e = 0; e < 8; ++e) v[nb][e] = v[nb][e] * t[nb][e] * u[nb][e];
            }
#pragma unroll
            for (int nb = 0; nb < C::NB; ++nb)
#pragma unroll
                for (int i = 8 * h; i < 8 * h + 8; i += 2) {
                    const float v0 = v[nb][i - 8 * h], v1 = v[nb][i + 1 - 8 * h];
                    const uint32_t pk = pack_bf16x2_hw(v0, v1);
                    const int r = 8 * ((i >> 2) - 2 * h) + 4 * (lane >> 5) + (i & 3);
                    const int c = nb * 32 + l32;
                    st[r * C::SROW + c] = (uint16_t)pk;
                    st[(r + 1) * C::SROW + c] = (uint16_t)(pk >> 16);
                }
            // the wave reads back only what it wrote (LDS operations of a wave
            // complete in order), then the next half block reuses the area
#pragma unroll
            for (int k = 0; k < 16 * C::CPR / 64; ++k) {
                const int c = lane + 64 * k;
                const int rr = c / C::CPR, cc = c % C::CPR;
                const int gm = row0 + dma_arow<C>(wm, mb) + 16 * h + rr, gn = col0 + cc * 8;
                const uint4 v = *(const uint4*)(st + rr * C::SROW + cc * 8);
                if (gm < tc.m_end && gn < p.N) {
                    if constexpr (FOLD) store_coherent(p.C + (size_t)gm * p.N + gn, v);
                    else *(uint4*)(p.C + (size_t)gm * p.N + gn) = v;
                }
            }
        }
    }
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (FOLD) {
        static_assert(!GATED && C::WTN == 128, "the fold works on the down projection's 128-column wave tiles");
        wait_vmcnt<0>();  // this wave's y stores are complete at the coherence point
        fold_rows<C>(p, tc, wm, col0, lane);
    }
}

// Work of P persistent workgroups: F rounds of one tile each (round r, tile
// r*P + w; the last round may be partial), then, split by K-steps, the tiles
// [F*P, total): each workgroup gets `share` consecutive K-steps of those.
// The split moves two fp32 tile pieces per workgroup through memory and
// restarts the pipeline per piece, so it is used (with a workspace) only when
// whole tiles would leave the workgroups idle for more than min_idle K-steps
// on average (the caller's threshold, kSkMinIdle by default).
constexpr int kSkMinIdle = 48;
constexpr int kSkMinShare = 8;  // K-steps: the shortest piece worth a pipeline restart
struct SkSplit {
    int F, W, share;
};
__device__ __forceinline__ SkSplit sk_split(int total, int nk, int P, bool can_split, int min_idle) {
    SkSplit k;
    const int rounds = ceil_div(total, P);
    const int64_t idle = (int64_t)(rounds * P - total) * nk;  // K-steps, summed over workgroups
    if (!can_split || total == 0 || idle <= (int64_t)min_idle * P) {
        k.F = rounds;
        k.W = 0;
        k.share = 1;
    } else {
        // split only the last partial round when its K-steps still give every
        // workgroup a piece of kSkMinShare or more (fewer split tiles, fewer
        // pieces through memory); otherwise the last one to two rounds
        const int full = total / P;
        const int64_t rest = (int64_t)(total - full * P) * nk;
        k.F = rest >= (int64_t)kSkMinShare * P ? full : max(0, full - 1);
        k.W = (total - k.F * P) * nk;
        k.share = ceil_div(k.W, P);
    }
    return k;
}

template <bool GATED, bool SK, bool FOLD = false>
__global__ __launch_bounds__(kGemmThreads, 1) void grouped_gemm_dma_kernel(GemmParams p, char* ws) {
    using C = DmaCfg<GATED>;
    __shared__ __align__(16) char smem[C::SMEM];
    const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
    const TileSched ts = tile_sched(p, smem + C::SCHED_OFF, C::BM, C::BN);
    const int total = ts.total_mt * ts.NT;
    const int nk = p.K / C::BK;
    f32x16 acc[C::NMAT][C::MB][C::NB];
    DmaSrc<C> src;
    if constexpr (!SK) {
        const int L = xcd_swizzle(blockIdx.x, gridDim.x);
        if (L >= total) return;
        const TileCoord tc = tile_coord(ts, p.n_seg, L, C::BM, C::BN);
        dma_sources<C, GATED>(src, p, tc, wave, lane);
        zero_acc<C>(acc);
        ksteps_prologue<C>(src, smem, 0, nk, wave);
        tile_ksteps<C, GATED>(acc, src, smem, 0, nk, wave, lane, kAfterNone, 0, p, tc, 0, 0);
        store_tile<C, GATED, FOLD>(acc, p, tc, smem, wave, lane);
    } else {
        const int P = gridDim.x;
        const int pw = xcd_swizzle(blockIdx.x, P);
        const SkSplit sk = sk_split(total, nk, P, ws != nullptr, p.sk_min_idle);
        // work items: full rounds (one tile each), then this workgroup's share
        // of the remaining K-steps; one loop so every stage is inlined once
        const int i0 = min(sk.W, pw * sk.share), i1 = min(sk.W, i0 + sk.share);
        int r = 0, i = i0;
        // the next work item (L < 0: none left)
        auto next_item = [&](int& L, int& ka, int& kb, int& slot) {
            slot = -1;
            while (r < sk.F) {
                L = r * P + pw;
                ka = 0;
                kb = nk;
                ++r;
                if (L < total) return;  // the last whole-tile round may be partial
            }
            if (i < i1) {
                const int t = i / nk;
                ka = i - t * nk;
                kb = min(nk, ka + (i1 - i));
                L = sk.F * P + t;
                // slot 0: the piece that starts the share, slot 1: the one that ends it
                if (ka != 0 || kb != nk) slot = i == i0 ? 0 : 1;
                i += kb - ka;
                return;
            }
            L = -1;
        };
        // The next item's first two K-steps are copied during this item's
        // last two (tile_ksteps), so they land while this item's results go
        // out and the pipeline does not drain between items.
        int L, ka, kb, slot;
        next_item(L, ka, kb, slot);
        TileCoord tc;
        if (L >= 0) {
            tc = tile_coord(ts, p.n_seg, L, C::BM, C::BN);
            dma_sources<C, GATED>(src, p, tc, wave, lane);
            ksteps_prologue<C>(src, smem, ka, kb, wave);
        }
        int after = kAfterNone, s0 = 0;
        while (L >= 0) {
            zero_acc<C>(acc);
            int L2, ka2, kb2, slot2;
            next_item(L2, ka2, kb2, slot2);
            TileCoord tc2 = tc;
            if (L2 >= 0) tc2 = tile_coord(ts, p.n_seg, L2, C::BM, C::BN);
            tile_ksteps<C, GATED>(acc, src, smem, ka, kb, wave, lane, after, s0, p, tc2, ka2, L2 >= 0 ? kb2 : ka2);
            store_tile<C, GATED, FOLD>(acc, p, tc, smem, wave, lane,
                                       slot < 0 ? nullptr : ws + ((size_t)2 * pw + slot) * kSkSlotBytes);
            after = kAfterStores;
            s0 = (s0 + kb - ka) & 1;
            L = L2;
            ka = ka2;
            kb = kb2;
            slot = slot2;
            tc = tc2;
        }
    }
}

// Sums the pieces of every tile that the stream-K split cut, in K order,
// then applies the epilogue. P persistent workgroups take the work items
// (split tile, slice) in turn: a tile of the split range is split when a
// share boundary falls strictly inside it, and a slice is one of kFixSplit
// parts of the tile's accumulator slots, so a split tile is finished by
// kFixSplit workgroups at once. Each thread adds its float4 slots of the
// pieces in the order of the pieces, as the unsplit path would (eight
// pieces' loads in flight), and writes its four rows of one column straight
// to the output.
constexpr int kFixSplit = 32;
constexpr int kFixInflight = 8;

template <bool GATED>
__global__ __launch_bounds__(kGemmThreads) void gemm_fixup_kernel(GemmParams p, const char* ws, int P) {
    using C = DmaCfg<GATED>;
    __shared__ __align__(16) char sched[C::SCHED];
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    // the tile count first, by a plain sum: with nothing split every
    // workgroup leaves before the schedule's scan
    __shared__ int s_wsum[kGemmThreads / 64];
    int cnt = 0;
    if (tid < p.n_seg) {
        const int beg = min(max(p.offsets[tid], 0), p.rows_cap);
        const int end = min(max(p.offsets[tid + 1], beg), p.rows_cap);
        cnt = ceil_div(end - beg, C::BM);
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) cnt += __shfl_xor(cnt, off);
    if (lane == 0) s_wsum[wave] = cnt;
    __syncthreads();
    const int total_mt = s_wsum[0] + s_wsum[1] + s_wsum[2] + s_wsum[3];
    const int nk = p.K / C::BK;
    const SkSplit sk = sk_split(total_mt * ceil_div(p.N, C::BN), nk, P, true, p.sk_min_idle);
    const int nsplit = sk.W / nk;  // tiles of the split range
    if (nsplit == 0 || (int)blockIdx.x >= nsplit * kFixSplit) return;
    const TileSched ts = tile_sched(p, sched, C::BM, C::BN);
    constexpr int NQ = C::MB * C::NB * 4;  // float4 slots of one matrix per thread
    static_assert(NQ % kFixSplit == 0, "slices of whole slots");
    constexpr int QPER = NQ / kFixSplit;
    const int wm = wave >> 1, wn = wave & 1;
    for (int item = blockIdx.x; item < nsplit * kFixSplit; item += gridDim.x) {
        const int t = item / kFixSplit, qs = item % kFixSplit;
        // the first share boundary after the tile's start
        const int q = (t * nk / sk.share + 1) * sk.share;
        if (q >= (t + 1) * nk) continue;  // no boundary inside: computed whole
        const int p0 = t * nk / sk.share, p1 = ((t + 1) * nk - 1) / sk.share;
        const TileCoord tc = tile_coord(ts, p.n_seg, sk.F * P + t, C::BM, C::BN);
        float4 sum[QPER][C::NMAT];
#pragma unroll
        for (int k = 0; k < QPER; ++k)
#pragma unroll
            for (int mat = 0; mat < C::NMAT; ++mat) sum[k][mat] = make_float4(0.f, 0.f, 0.f, 0.f);
        auto piece = [&](int pw) {
            const int slot = pw * sk.share >= t * nk ? 0 : 1;  // share starts inside tile t, or ends in it
            return (const float4*)(ws + ((size_t)2 * pw + slot) * kSkSlotBytes);
        };
        auto add = [&](float4& a, const float4& v) {
            a.x += v.x;
            a.y += v.y;
            a.z += v.z;
            a.w += v.w;
        };
        int pw = p0;
        for (; pw + kFixInflight - 1 <= p1; pw += kFixInflight) {
            float4 v[kFixInflight][QPER][C::NMAT];
#pragma unroll
            for (int j = 0; j < kFixInflight; ++j) {
                const float4* d = piece(pw + j);
#pragma unroll
                for (int k = 0; k < QPER; ++k)
#pragma unroll
                    for (int mat = 0; mat < C::NMAT; ++mat)
                        v[j][k][mat] = d[(mat * NQ + qs * QPER + k) * kGemmThreads + tid];
            }
#pragma unroll
            for (int j = 0; j < kFixInflight; ++j)
#pragma unroll
                for (int k = 0; k < QPER; ++k)
#pragma unroll
                    for (int mat = 0; mat < C::NMAT; ++mat) add(sum[k][mat], v[j][k][mat]);
        }
        for (; pw <= p1; ++pw) {
            const float4* d = piece(pw);
#pragma unroll
            for (int k = 0; k < QPER; ++k)
#pragma unroll
                for (int mat = 0; mat < C::NMAT; ++mat)
                    add(sum[k][mat], d[(mat * NQ + qs * QPER + k) * kGemmThreads + tid]);
        }
#pragma unroll
        for (int k = 0; k < QPER; ++k) {
            const int qq = qs * QPER + k;  // slot (mb, nb, i4) in the order of store_piece
            const int i4 = qq & 3, nb = (qq >> 2) % C::NB, mb = (qq >> 2) / C::NB;
            const int r0 = dma_arow<C>(wm, mb) + 8 * i4 + 4 * (lane >> 5);
            const int gn = tc.n0 + wn * C::WTN + nb * 32 + (lane & 31);
            const float g4[4] = {sum[k][0].x, sum[k][0].y, sum[k][0].z, sum[k][0].w};
            const float4 u = sum[k][C::NMAT - 1];
            const float u4[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const float v = GATED ? silu_mul(g4[j], u4[j]) : g4[j];
                const int gm = tc.m0 + r0 + j;
                if (gm < tc.m_end && gn < p.N) p.C[(size_t)gm * p.N + gn] = (uint16_t)pack_bf16x2_hw(v, 0.f);
            }
        }
    }
}

// CUs of the current device, rounded down to a multiple of 8 (XCD deal)
static int stream_k_workgroups() {
    static int cached[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
    if (cached[dev] == 0) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
        cached[dev] = n / 8 * 8;
    }
    return cached[dev];
}

template <bool GATED>
hipError_t launch_gemm_dma(const GemmParams& g0, void* ws, size_t ws_bytes, hipStream_t s) {
    using C = DmaCfg<GATED>;
    GemmParams g = g0;
    g.sk_min_idle = g0.sk_min_idle < 0 ? kSkMinIdle : g0.sk_min_idle;
    // persistent: one workgroup per CU, each XCD a contiguous range of tiles
    const int P = stream_k_workgroups();
    if constexpr (!GATED) {
        if (g.fold.out != nullptr) {
            // the fold needs every tile whole (no stream-K pieces)
            if (P <= 0) return hipErrorInvalidValue;
            hipLaunchKernelGGL((grouped_gemm_dma_kernel<false, true, true>), dim3(P), dim3(kGemmThreads), 0, s, g,
                               (char*)nullptr);
            return hipGetLastError();
        }
    }
    if (P > 0) {
        const bool split = ws != nullptr && ws_bytes >= (size_t)2 * P * kSkSlotBytes;
        hipLaunchKernelGGL((grouped_gemm_dma_kernel<GATED, true>), dim3(P), dim3(kGemmThreads), 0, s, g,
                           split ? (char*)ws : (char*)nullptr);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess || !split) return e;
        hipLaunchKernelGGL((gemm_fixup_kernel<GATED>), dim3(P), dim3(kGemmThreads), 0, s, g, (const char*)ws, P);
        return hipGetLastError();
    }
    const int64_t mt_max = ceil_div64(g.rows_cap, C::BM) + g.n_seg;
    const int64_t nt = ceil_div64(g.N, C::BN);
    int64_t blocks = (mt_max * nt + 7) / 8 * 8;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
    hipLaunchKernelGGL((grouped_gemm_dma_kernel<GATED, false>), dim3((unsigned)blocks), dim3(kGemmThreads), 0, s, g,
                       (char*)nullptr);
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
                                                             int n_seg, int rows_cap, int d, int d_ff,
                                                             const int32_t* __restrict__ a_rows, int a_count) {
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (idx >= (int64_t)rows_cap * d_ff) return;
    const int row = (int)(idx / d_ff), j = (int)(idx % d_ff);
    const int s = find_segment(offsets, n_seg, rows_cap, row);
    if (s < 0) return;
    const float* ar = a + (size_t)gathered_row(a_rows, a_count, row) * d;
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

size_t ffn_workspace_bytes() {
    const int P = stream_k_workgroups();
    return P > 0 ? (size_t)2 * P * kSkSlotBytes : 0;
}

// Workgroup tile of the bf16 grouped GEMMs (batches above the skinny
// kernels' size). When d and d_ff are whole 64-column K-steps, the persistent
// 256-row kernel with direct-to-LDS copies runs at any group size: from 80
// rows per group up it measured 1.5-2.4x faster than 128-row register-staged
// tiles, the padding of each group to whole 256-row tiles included. Otherwise
// the register-staged kernels: 256-row tiles (128x128 per wave, half the LDS
// traffic per MFMA) when groups average 1024 rows or more, else 128-row.
enum { kTile128 = 0, kTile256 = 1, kTileDma = 2 };
constexpr bool kFdb256 = false;  // no registers left for a second fragment set
static int ffn_tile(const FfnArgs& a) {
    if (a.d % kDmaBK == 0 && a.d_ff % kDmaBK == 0) return kTileDma;
    return (int64_t)a.rows_cap < (int64_t)1024 * a.n_seg ? kTile128 : kTile256;
}

bool ffn_can_fold(const FfnArgs& a) {
    return a.dtype == BMOE_BF16 && a.rows_cap > 0 && !ffn_skinny_fits(a) && ffn_tile(a) == kTileDma &&
           a.d % 128 == 0 && stream_k_workgroups() > 0;
}

hipError_t launch_ffn(const FfnArgs& a, hipStream_t s, int part) {
    if (a.rows_cap == 0) return hipSuccess;
    const bool up = part != 2, down = part != 1;
    if (a.dtype == BMOE_F32) {
        const int64_t n1 = (int64_t)a.rows_cap * a.d_ff, n2 = (int64_t)a.rows_cap * a.d;
        if (up) {
            hipLaunchKernelGGL(ffn_f32_gateup_kernel, dim3((unsigned)ceil_div64(n1, 256)), dim3(256), 0, s,
                               (const float*)a.a, (const float*)a.w_gate, (const float*)a.w_up, (float*)a.h,
                               a.offsets, a.n_seg, a.rows_cap, a.d, a.d_ff, a.a_rows, a.a_count);
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
    if (ffn_skinny_fits(a)) return launch_ffn_skinny(a, s, part);
    const int tile = ffn_tile(a);
    if (up) {
        GemmParams g1{(const uint16_t*)a.a, (const uint16_t*)a.w_gate, (const uint16_t*)a.w_up,
                      (uint16_t*)a.h, a.offsets, a.n_seg, a.rows_cap, a.d_ff, a.d};
        g1.a_rows = a.a_rows;
        g1.a_count = a.a_count;
        g1.sk_min_idle = a.split_min_idle;
        hipError_t e = tile == kTileDma   ? launch_gemm_dma<true>(g1, a.ws, a.ws_bytes, s)
                       : tile == kTile256 ? launch_gemm<true, 256, 128, 64, kFdb256>(g1, s)
                                          : launch_gemm<true, 128, 128, 64, true>(g1, s);
        if (e != hipSuccess) return e;
    }
    if (down) {
        GemmParams g2{(const uint16_t*)a.h, (const uint16_t*)a.w_down, nullptr, (uint16_t*)a.y,
                      a.offsets, a.n_seg, a.rows_cap, a.d, a.d_ff};
        g2.sk_min_idle = a.split_min_idle;
        g2.fold = a.fold;
        return tile == kTileDma   ? launch_gemm_dma<false>(g2, a.ws, a.ws_bytes, s)
               : tile == kTile256 ? launch_gemm<false, 256, 256, 64, kFdb256>(g2, s)
                                  : launch_gemm<false, 128, 256, 64, true>(g2, s);
    }
    return hipSuccess;
}

}  // namespace bmoe
