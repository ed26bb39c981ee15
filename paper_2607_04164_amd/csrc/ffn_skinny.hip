// Skinny grouped GEMMs for decode-sized batches: the per-united-expert
// SwiGLU FFN of Sec. 2.1 when every group holds only a few dozen rows, so the
// layer is bound by streaming the united-expert weights, not by MFMA. Two
// kernels share the grid and the MFMA layout: skinny_dma_kernel (further
// down) copies every operand straight into LDS and runs whenever K is a
// multiple of 64; skinny_gemm_kernel, described here, stages operands through
// registers and takes any K.
//
// One workgroup (4 waves) owns one segment and 64 output columns; wave w owns
// columns n0 .. n0+15 with n0 = 64*cb + 16*w (for the fused gate/up GEMM: those
// rows of both W_gate and W_up). The segment's rows are taken 64 at a time
// (one pass over the weights per 64 rows). Per K-chunk of 256 columns:
//   - the 64 activation rows (clamped to the segment) are loaded to registers
//     and written to a swizzled LDS slot that the four waves share;
//   - each wave loads its weight rows straight into registers in the MFMA
//     operand layout (each load instruction reads 64 contiguous bytes of each
//     of the wave's 16 weight rows);
//   - 16x16x32 bf16 MFMA with the weights as the A operand and the
//     activations as the B operand, D[weight row][row of the segment].
// MFMA u covers columns 32u .. 32u+31 of the chunk, lane group q its columns
// 32u + 8q .. 32u + 8q + 7 (both operands). Chunks are double-buffered in
// registers and LDS; the loop is unrolled by two so that no register array is
// indexed at run time, and chunks past the end hold zero activations instead
// of branching around MFMAs.
#include "bmoe_common.h"

namespace bmoe {
namespace {

constexpr int kSkThreads = 256;
constexpr int kSkRows = 64;                      // activation rows per pass
constexpr int kSkKC = 256;                       // K columns per chunk
constexpr int kSkCols = 64;                      // output columns per workgroup
constexpr int kSkRowBytes = kSkKC * 2;           // 512 B per LDS row
constexpr int kSkSlot = kSkRows * kSkRowBytes;   // 32 KiB per chunk
constexpr int kSkXLoads = kSkSlot / 16 / kSkThreads;  // 16-byte activation loads per thread

typedef uint32_t v4u __attribute__((ext_vector_type(4)));  // native vector: stays in registers

struct SkinnyParams {
    const uint16_t* A;   // [rows_cap, K]
    const uint16_t* B0;  // [n_seg, N, K]
    const uint16_t* B1;  // [n_seg, N, K] (gated: W_up)
    uint16_t* C;         // [rows_cap, N]
    const int32_t* offsets;
    int n_seg, rows_cap, N, K;
    const int32_t* a_rows = nullptr;  // gathered A: row r is A[a_rows[r]] (A has a_count rows)
    int a_count = 0;
};

// LDS byte offset of logical 16-byte chunk c of activation row r
__device__ __forceinline__ int sk_off(int r, int c) { return r * kSkRowBytes + ((c ^ (r & 15)) << 4); }

// Chunk c of the pass's activation rows (source rows xrow, see the kernel)
// into xs, and of the lane's weight rows into wv. Addresses past the end of a
// row or past the last chunk are clamped to column 0 (finite values); the
// activations of those columns are zeroed when they are written to LDS, so
// their products vanish and no load result is touched before it is used.
template <int NMAT>
__device__ __forceinline__ void sk_load(const SkinnyParams& p, const uint16_t* const (&wp)[NMAT], int c, int nch,
                                        const int (&xrow)[kSkXLoads], int q, v4u (&xs)[kSkXLoads],
                                        v4u (&wv)[NMAT][8]) {
    const int K = p.K;
    const int kc0 = min(c, nch - 1) * kSkKC;
#pragma unroll
    for (int j = 0; j < kSkXLoads; ++j) {
        const int i = threadIdx.x + kSkThreads * j;
        int col = kc0 + (i & 31) * 8;
        if (col >= K) col = 0;
        xs[j] = *(const v4u*)(p.A + (size_t)xrow[j] * K + col);
    }
    // the activations are issued before the weights: their LDS store (one
    // chunk earlier than the weights' MFMAs) then waits only for older loads
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int mat = 0; mat < NMAT; ++mat)
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int col = kc0 + u * 32 + q * 8;
            wv[mat][u] = *(const v4u*)(wp[mat] + (col < K ? col : 0));
        }
}

__device__ __forceinline__ void sk_store_x(const v4u (&xs)[kSkXLoads], char* slot, int c, int nch, int K) {
    const int kc0 = c * kSkKC;
#pragma unroll
    for (int j = 0; j < kSkXLoads; ++j) {
        const int i = threadIdx.x + kSkThreads * j;
        const uint32_t keep = (c < nch && kc0 + (i & 31) * 8 < K) ? ~0u : 0u;
        *(v4u*)(slot + sk_off(i >> 5, i & 31)) = xs[j] & keep;
    }
}

template <int NMAT>
__device__ __forceinline__ void sk_compute(f32x4 (&acc)[NMAT][4], const char* slot, const v4u (&wv)[NMAT][8],
                                           int r16, int q) {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        v4u xf[4];
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) xf[nt] = *(const v4u*)(slot + sk_off(nt * 16 + r16, u * 4 + q));
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
#pragma unroll
            for (int mat = 0; mat < NMAT; ++mat)
                acc[mat][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, wv[mat][u]),
                                                                       __builtin_bit_cast(bf16x8, xf[nt]),
                                                                       acc[mat][nt], 0, 0, 0);
    }
}

template <bool GATED>
__global__ __launch_bounds__(kSkThreads, 1) void skinny_gemm_kernel(SkinnyParams p) {
    constexpr int NMAT = GATED ? 2 : 1;
    __shared__ __align__(16) char lds[2 * kSkSlot];
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int ncb = ceil_div(p.N, kSkCols);
    const int s = blockIdx.x / ncb, cb = blockIdx.x % ncb;
    if (s >= p.n_seg) return;
    const int beg = min(max(p.offsets[s], 0), p.rows_cap);
    const int end = min(max(p.offsets[s + 1], beg), p.rows_cap);
    if (end <= beg) return;
    const int K = p.K, N = p.N;
    const int nch = ceil_div(K, kSkKC);
    const int r16 = lane & 15, q = lane >> 4;
    const int n0 = cb * kSkCols + wave * 16;
    const int wrow = min(n0 + r16, N - 1);  // clamped: loads stay in bounds
    const uint16_t* wp[NMAT];
    wp[0] = p.B0 + ((size_t)s * N + wrow) * K;
    if constexpr (GATED) wp[NMAT - 1] = p.B1 + ((size_t)s * N + wrow) * K;
    char* slot0 = lds;
    char* slot1 = lds + kSkSlot;

    for (int m0 = beg; m0 < end; m0 += kSkRows) {
        f32x4 acc[NMAT][4];
#pragma unroll
        for (int mat = 0; mat < NMAT; ++mat)
#pragma unroll
            for (int nt = 0; nt < 4; ++nt) acc[mat][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
        // two stages: chunk c's weights are loaded two chunks ahead, its
        // activations one chunk before they are written to LDS (a third stage
        // measured slower)
        // source rows of this thread's activation loads: the pass's rows
        // [m0, m0+64) clamped to the segment, gathered when A is
        int xrow[kSkXLoads];
#pragma unroll
        for (int j = 0; j < kSkXLoads; ++j)
            xrow[j] = gathered_row(p.a_rows, p.a_count, min(m0 + ((tid + kSkThreads * j) >> 5), end - 1));
        v4u xs0[kSkXLoads], xs1[kSkXLoads];
        v4u w0[NMAT][8], w1[NMAT][8];
        sk_load<NMAT>(p, wp, 0, nch, xrow, q, xs0, w0);
        sk_load<NMAT>(p, wp, 1, nch, xrow, q, xs1, w1);
        sk_store_x(xs0, slot0, 0, nch, K);
        __syncthreads();
        for (int c = 0; c < nch; c += 2) {
            sk_compute<NMAT>(acc, slot0, w0, r16, q);  // chunk c
            sk_store_x(xs1, slot1, c + 1, nch, K);     // chunk c+1 (slot released by the last barrier)
            sk_load<NMAT>(p, wp, c + 2, nch, xrow, q, xs0, w0);
            __syncthreads();
            sk_compute<NMAT>(acc, slot1, w1, r16, q);  // chunk c+1 (zero activations past the end)
            sk_store_x(xs0, slot0, c + 2, nch, K);     // chunk c+2
            sk_load<NMAT>(p, wp, c + 3, nch, xrow, q, xs1, w1);
            __syncthreads();
        }

        // epilogue: lane holds D[weight row 4q+i][segment row r16] of every
        // row tile nt, i.e. output columns n0+4q .. n0+4q+3 of row m0+16nt+r16
        const int col = n0 + 4 * q;
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
            const int row = m0 + nt * 16 + r16;
            if (row >= end) continue;
            float v[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                if constexpr (GATED) v[i] = silu_mul(acc[0][nt][i], acc[NMAT - 1][nt][i]);
                else v[i] = acc[0][nt][i];
            }
            uint16_t* dst = p.C + (size_t)row * N + col;
            if (col + 3 < N) {
                *(uint2*)dst = make_uint2(pack_bf16x2_hw(v[0], v[1]), pack_bf16x2_hw(v[2], v[3]));
            } else {
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (col + i < N) dst[i] = f32_to_bf16(v[i]);
            }
        }
        // the LDS slots are rewritten by the next pass
        __syncthreads();
    }
}

// ---- the same FFN with every operand copied straight into LDS (K % 64 == 0)
//
// The register-staged kernel above keeps about two chunks of weights in
// flight per wave, and its activation stores wait for loads issued one
// chunk earlier, so each chunk waits for most of a memory latency. Here the
// activation rows and the workgroup's weight rows of a 64-column chunk are
// copied with global_load_lds (one 128-byte line per row and copy row, 1 KB
// per instruction) into a ring of slots, up to NSL-2 chunks ahead of the two
// being multiplied, and both MFMA operands are read from LDS. A slot row's
// 16-byte pieces are XOR-swizzled by (row & 7), so the 8 rows of a read
// group fall on different banks. One barrier per two chunks: after it every
// wave's copies of both have landed and every wave has finished reading the
// slots the next copies overwrite. Decode-shaped (8 segments, d = 2048,
// d_ff = 1408): gate/up 26 -> 21 us, down 14.0 -> 13.5 us with one barrier
// per chunk, then 18.0 and 11.6 us with two (the copy loop alone streams the
// weights at the rate of plain streaming probes; the fragment reads and
// MFMAs between barriers were what it lost). Reading the next chunk's
// fragments during the current chunk's MFMAs measured slower.
constexpr int kS2KC = 64;             // K columns per chunk
constexpr int kS2RowB = kS2KC * 2;    // bytes per slot row (one 128-byte line)

template <int NMAT>
struct S2Cfg {
    static constexpr int ROWS = kSkRows + NMAT * kSkCols;  // activation rows, then each matrix's weight rows
    static constexpr int SLOT = ROWS * kS2RowB;            // 16 KB (down) / 24 KB (gate/up)
    static constexpr int NSL = NMAT == 2 ? 6 : 8;            // 144 KB / 128 KB of LDS
    static constexpr int CPB = 2;                            // chunks per barrier
    static constexpr int NDMA = ROWS / 8;                    // copy instructions per chunk
    static constexpr int DPW = NDMA / 4;                     // per wave
    static_assert(NDMA % 4 == 0 && kSkRows % 64 == 0 && kSkCols % 64 == 0, "copy rows split evenly");
    static_assert(NSL - 2 * CPB >= 0 && NSL - 2 * CPB <= 7, "run-time copy wait covers 0..7 later chunks");
    static_assert(NSL * SLOT <= 160 * 1024, "LDS of one workgroup");
};

__device__ __forceinline__ int s2_off(int row, int chunk) { return row * kS2RowB + ((chunk ^ (row & 7)) << 4); }

template <bool GATED>
__global__ __launch_bounds__(kSkThreads, 1) void skinny_dma_kernel(SkinnyParams p) {
    constexpr int NMAT = GATED ? 2 : 1;
    using C = S2Cfg<NMAT>;
    __shared__ __align__(16) char lds[C::NSL * C::SLOT];
    // the wave index in an SGPR: the copy bases below stay scalar
    const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
    const int ncb = ceil_div(p.N, kSkCols);
    const int s = blockIdx.x / ncb, cb = blockIdx.x % ncb;
    if (s >= p.n_seg) return;
    const int beg = min(max(p.offsets[s], 0), p.rows_cap);
    const int end = min(max(p.offsets[s + 1], beg), p.rows_cap);
    if (end <= beg) return;
    const int K = p.K, N = p.N;
    const int nch = K / kS2KC;
    const int n0 = cb * kSkCols;
    const int r16 = lane & 15, q = lane >> 4;
    const uint32_t lds0 = (uint32_t)(uintptr_t)lds;

    // copy instruction i of this wave fills slot rows [8g, 8g+8), g = wave*DPW + i:
    // rows [0, 64) are activation rows, then 64 weight rows of each matrix
    const char* base[C::DPW];
    uint32_t off[C::DPW];
    int lane_v = lane;
    asm volatile("" : "+v"(lane_v));  // keep the per-lane parts from being hoisted and spilled
    const int lrow = lane_v >> 3, lchk = lane_v & 7;
#pragma unroll
    for (int i = 0; i < C::DPW; ++i) {
        const int g = wave * C::DPW + i;
        const int region = g >> 3;  // 0: activations, 1 + mat: weights of matrix mat
        const int row = 8 * g + lrow;
        if (region > 0) {
            const uint16_t* w = (GATED && region == 2) ? p.B1 : p.B0;
            base[i] = (const char*)(w + ((size_t)s * N + n0) * K);
            const int wr = min(n0 + (row - 64 * region), N - 1) - n0;
            off[i] = (uint32_t)((size_t)wr * K * 2 + ((lchk ^ (row & 7)) << 4));
        } else {
            base[i] = (const char*)p.A;
            off[i] = 0;  // set per pass
        }
    }
    auto issue = [&](int c) {
        const uint32_t slot = lds0 + (uint32_t)((c % C::NSL) * C::SLOT);
#pragma unroll
        for (int i = 0; i < C::DPW; ++i)
            dma16s(base[i] + (size_t)c * kS2RowB, off[i], slot + (uint32_t)((wave * C::DPW + i) * 1024));
    };

    for (int m0 = beg; m0 < end; m0 += kSkRows) {
        // source rows of the pass: [m0, m0+64) clamped to the segment, gathered when A is
#pragma unroll
        for (int i = 0; i < C::DPW; ++i) {
            const int g = wave * C::DPW + i;
            if ((g >> 3) == 0) {
                const int row = 8 * g + lrow;
                const int arow = gathered_row(p.a_rows, p.a_count, min(m0 + row, end - 1));
                off[i] = (uint32_t)((size_t)arow * K * 2 + ((lchk ^ (row & 7)) << 4));
            }
        }
        f32x4 acc[NMAT][4];
#pragma unroll
        for (int mat = 0; mat < NMAT; ++mat)
#pragma unroll
            for (int nt = 0; nt < 4; ++nt) acc[mat][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
        // The MFMAs of chunk c (the A operand: the weights, the B operand: the
        // activation rows), from its ring slot.
        auto chunk_mfmas = [&](int c) {
            const char* sl = lds + (c % C::NSL) * C::SLOT;
#pragma unroll
            for (int kk = 0; kk < 2; ++kk) {
                v4u wv[NMAT], xv[4];
#pragma unroll
                for (int mat = 0; mat < NMAT; ++mat) {
                    const int row = kSkRows + mat * kSkCols + wave * 16 + r16;
                    wv[mat] = *(const v4u*)(sl + s2_off(row, kk * 4 + q));
                }
#pragma unroll
                for (int nt = 0; nt < 4; ++nt) xv[nt] = *(const v4u*)(sl + s2_off(nt * 16 + r16, kk * 4 + q));
#pragma unroll
                for (int nt = 0; nt < 4; ++nt)
#pragma unroll
                    for (int mat = 0; mat < NMAT; ++mat)
                        acc[mat][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, wv[mat]),
                                                                               __builtin_bit_cast(bf16x8, xv[nt]),
                                                                               acc[mat][nt], 0, 0, 0);
            }
        };
        // Prologue: the first NSL - CPB chunks. Each step then waits for its
        // CPB chunks and, after one barrier, refills the slots of the previous
        // step's chunks. A step's chunks run without a branch between them, so
        // the compiler can issue all their fragment reads and MFMAs as one
        // block (two chunks per barrier: the decode-shaped gate/up 20.8 ->
        // 17.6 us, down 14.0 -> 11.6 us with the chunk count known at compile
        // time in a stand-alone harness); an odd last chunk takes a step of
        // its own.
        for (int c = 0; c < C::NSL - C::CPB && c < nch; ++c) issue(c);
        const int nsteps = nch - nch % C::CPB;
        for (int c0 = 0; c0 < nsteps; c0 += C::CPB) {
            // this wave's copies of the step's chunks are done when at most the
            // later chunks' copies are outstanding; after the barrier every
            // wave's are, and no wave still reads the previous step's slots
            wait_vmcnt_rt<C::DPW>(min(C::NSL - C::CPB, nch - c0) - C::CPB);
            lds_reads_done();
            wg_barrier();
#pragma unroll
            for (int j = 0; j < C::CPB; ++j)
                if (c0 + C::NSL - C::CPB + j < nch) issue(c0 + C::NSL - C::CPB + j);
#pragma unroll
            for (int j = 0; j < C::CPB; ++j) chunk_mfmas(c0 + j);
        }
        if (nsteps < nch) {  // every copy was issued; wait for all of them
            wait_vmcnt<0>();
            lds_reads_done();
            wg_barrier();
            for (int c = nsteps; c < nch; ++c) chunk_mfmas(c);
        }

        // epilogue: lane holds D[weight row 4q+i][segment row r16] of every
        // row tile nt, i.e. output columns col .. col+3 of row m0+16nt+r16
        const int col = n0 + wave * 16 + 4 * q;
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
            const int row = m0 + nt * 16 + r16;
            if (row >= end) continue;
            float v[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                if constexpr (GATED) v[i] = silu_mul(acc[0][nt][i], acc[NMAT - 1][nt][i]);
                else v[i] = acc[0][nt][i];
            }
            uint16_t* dst = p.C + (size_t)row * N + col;
            if (col + 3 < N) {
                *(uint2*)dst = make_uint2(pack_bf16x2_hw(v[0], v[1]), pack_bf16x2_hw(v[2], v[3]));
            } else {
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (col + i < N) dst[i] = f32_to_bf16(v[i]);
            }
        }
        // the ring is refilled by the next pass: every read done, and the
        // stores complete before its copies are counted
        wait_vmcnt<0>();
        lds_reads_done();
        wg_barrier();
    }
}

template <bool GATED>
hipError_t launch_skinny(const SkinnyParams& sp, hipStream_t s) {
    const int64_t blocks = (int64_t)sp.n_seg * ceil_div(sp.N, kSkCols);
    if (blocks <= 0) return hipSuccess;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
    // the copies address A rows by 32-bit byte offsets from A
    const int64_t a_rows = sp.a_rows ? sp.a_count : sp.rows_cap;
    if (sp.K % kS2KC == 0 && a_rows * sp.K * 2 < ((int64_t)1 << 31) && (int64_t)kSkCols * sp.K * 2 < ((int64_t)1 << 31))
        hipLaunchKernelGGL((skinny_dma_kernel<GATED>), dim3((unsigned)blocks), dim3(kSkThreads), 0, s, sp);
    else
        hipLaunchKernelGGL((skinny_gemm_kernel<GATED>), dim3((unsigned)blocks), dim3(kSkThreads), 0, s, sp);
    return hipGetLastError();
}

}  // namespace

bool ffn_skinny_fits(const FfnArgs& a) {
    return a.dtype == BMOE_BF16 && (int64_t)a.rows_cap <= (int64_t)kSkRows * a.n_seg;
}

hipError_t launch_ffn_skinny(const FfnArgs& a, hipStream_t s, int part) {
    const bool up = part != 2, down = part != 1;
    if (up) {
        SkinnyParams g1{(const uint16_t*)a.a, (const uint16_t*)a.w_gate, (const uint16_t*)a.w_up, (uint16_t*)a.h,
                        a.offsets, a.n_seg, a.rows_cap, a.d_ff, a.d};
        g1.a_rows = a.a_rows;
        g1.a_count = a.a_count;
        hipError_t e = launch_skinny<true>(g1, s);
        if (e != hipSuccess) return e;
    }
    if (down) {
        SkinnyParams g2{(const uint16_t*)a.h, (const uint16_t*)a.w_down, nullptr, (uint16_t*)a.y, a.offsets,
                        a.n_seg, a.rows_cap, a.d, a.d_ff};
        return launch_skinny<false>(g2, s);
    }
    return hipSuccess;
}

}  // namespace bmoe
