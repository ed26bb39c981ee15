// Internal helpers shared by the HIP kernels of libbrownout_moe (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "brownout_moe.h"

namespace bmoe {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;

constexpr int kWave = 64;

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float(((uint32_t)b) << 16);
}

// float -> bf16, round to nearest even (NaN stays NaN).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return (uint32_t)f32_to_bf16(lo) | ((uint32_t)f32_to_bf16(hi) << 16);
}

typedef __bf16 bf16x2_hw __attribute__((ext_vector_type(2)));
typedef float f32x2_hw __attribute__((ext_vector_type(2)));

// two floats -> packed bf16 (low, high) with the hardware round-to-nearest-even convert
__device__ __forceinline__ uint32_t pack_bf16x2_hw(float lo, float hi) {
    f32x2_hw v = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_hw));
}

// silu(g) * u = g / (1 + e^-g) * u with the hardware exp2 and reciprocal
// (relative error ~1e-7, far below the bf16 rounding that follows)
__device__ __forceinline__ float silu_mul(float g, float u) {
    return g * __builtin_amdgcn_rcpf(1.f + __expf(-g)) * u;
}

__device__ __forceinline__ bf16x8 as_bf16x8(const uint4& v) {
    return __builtin_bit_cast(bf16x8, v);
}

// 16x16x32 bf16 MFMA: lane l holds A[l%16][8*(l/16)+j], B[8*(l/16)+j][l%16];
// result D[4*(l/16)+i][l%16] in element i.
__device__ __forceinline__ f32x4 mfma16(const uint4& a, const uint4& b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
}

// 32x32x16 bf16 MFMA: lane l holds A[l%32][8*(l/32)+j], B[8*(l/32)+j][l%32];
// result D[8*(i/4)+4*(l/32)+i%4][l%32] in element i.
__device__ __forceinline__ f32x16 mfma32(const uint4& a, const uint4& b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
}

__host__ __device__ constexpr int ceil_div(int a, int b) { return (a + b - 1) / b; }
__host__ __device__ constexpr int64_t ceil_div64(int64_t a, int64_t b) { return (a + b - 1) / b; }

// ---- direct global->LDS loads and the waits that go with them
//
// global_load_lds_dwordx4: every lane copies 16 bytes from its global address
// to LDS at M0 + 16 * lane. Issued through inline asm because with the
// builtin the compiler waits for every outstanding copy before each LDS read
// and at each barrier; callers wait explicitly with wait_vmcnt / wg_barrier.
__device__ __forceinline__ void dma16(const void* gptr, uint32_t lds_addr) {
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(gptr), "s"(lds_addr)
                 : "memory", "m0");
}
// Same copy with a uniform 64-bit base in SGPRs and a 32-bit per-lane byte
// offset (the SADDR form): one VGPR per copy source instead of two.
// The base must be workgroup-uniform; readfirstlane makes that explicit (it
// folds away when the compiler already holds the base in SGPRs).
__device__ __forceinline__ void dma16s(const void* base, uint32_t voff, uint32_t lds_addr) {
    const uint64_t b = (uint64_t)(uintptr_t)base;
    const uint64_t ub = ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(b >> 32)) << 32) |
                        (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)b);
    asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(ub),
                 "s"(__builtin_amdgcn_readfirstlane(lds_addr))
                 : "memory", "m0");
}
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
// wait until at most PER*n of this wave's vector-memory operations are in flight (n in 0..7)
template <int PER>
__device__ __forceinline__ void wait_vmcnt_rt(int n) {
#define BMOE_VMW(m) wait_vmcnt<((m) * PER > 63 ? 63 : (m) * PER)>()
    switch (n < 0 ? 0 : n) {
        case 0: BMOE_VMW(0); break;
        case 1: BMOE_VMW(1); break;
        case 2: BMOE_VMW(2); break;
        case 3: BMOE_VMW(3); break;
        case 4: BMOE_VMW(4); break;
        case 5: BMOE_VMW(5); break;
        case 6: BMOE_VMW(6); break;
        default: BMOE_VMW(7); break;
    }
#undef BMOE_VMW
}
__device__ __forceinline__ void lds_reads_done() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
__device__ __forceinline__ void wg_barrier() { asm volatile("s_barrier" ::: "memory"); }

// Block-wide exclusive scan of up to 256 ints held one per thread (blockDim = 256).
// `buf` is 256 ints of LDS. Returns the exclusive prefix; *total gets the sum.
__device__ __forceinline__ int block_exclusive_scan_256(int v, int* buf, int* total) {
    const int tid = threadIdx.x;
    buf[tid] = v;
    __syncthreads();
    for (int off = 1; off < 256; off <<= 1) {
        int add = tid >= off ? buf[tid - off] : 0;
        __syncthreads();
        buf[tid] += add;
        __syncthreads();
    }
    int incl = buf[tid];
    *total = buf[255];
    __syncthreads();
    return incl - v;
}

}  // namespace bmoe

// Launchers implemented by the kernel files; arguments already validated.
namespace bmoe {

struct UnitedInitArgs {
    const int32_t* e2g;
    const void* src[3];  // member experts' W_gate, W_up [E, d_ff, d], W_down [E, d, d_ff]
    void* dst[3];        // united experts' [G, ...]
    int E, G, d, d_ff, dtype;
};
hipError_t launch_united_init(const UnitedInitArgs& a, hipStream_t s);

struct DistillArgs {
    const int32_t* e2g;
    const float* w;         // routing frequencies [E]
    const void* y_expert;   // [E*T, d]
    const void* y_united;   // [G*T, d]
    double* mse;            // [G]
    double* total;          // nullable
    void* ws;               // distill_blocks(G, T) * G doubles
    int E, G, T, d, dtype;
};
int distill_blocks(int G, int T);
hipError_t launch_distill_mse(const DistillArgs& a, hipStream_t s);

struct RouteArgs {
    const void* x;
    const void* w;
    const float* bias;
    const float* logits_in;
    const int32_t* e2g;
    int32_t* topk_idx;
    float* topk_w;
    int32_t* slot_group;
    float* slot_gate;
    float* logits_out;
    int T, d, E, k, G, norm, dtype;
};
hipError_t launch_route(const RouteArgs& a, hipStream_t s);

struct DispatchArgs {
    const int32_t* slot_group;
    const void* x;
    int32_t* counts;
    int32_t* offsets;
    int32_t* perm_token;
    int32_t* slot_row;
    void* x_perm;
    void* ws;
    int T, d, k, G, elem_bytes;
};
size_t dispatch_ws_bytes(int T, int G);
hipError_t launch_dispatch(const DispatchArgs& a, hipStream_t s);
// a.ws ignored: the library's own per-device array (BMOE_DISPATCH_SCRATCH_BYTES)
hipError_t launch_dispatch_noalloc(const DispatchArgs& a, hipStream_t s);

// Combine folded into the down projection (out == nullptr: not folded).
struct FoldArgs {
    const int32_t* perm_token = nullptr;  // [rows]: token of each row
    const int32_t* slot_row = nullptr;    // [T, k]
    const float* slot_gate = nullptr;     // [T, k]
    const uint16_t* y_shared = nullptr;   // [T, d] bf16 or nullptr
    uint16_t* out = nullptr;              // [T, d] bf16
    int32_t* cnt = nullptr;               // [T, d / 128] counters, zero between calls
    int k = 0;
};

struct FfnArgs {
    const int32_t* offsets;
    const void* a;
    const void* w_gate;
    const void* w_up;
    const void* w_down;
    void* h;
    void* y;
    void* ws;  // optional stream-K workspace (nullptr: one tile per workgroup)
    size_t ws_bytes;
    int n_seg, rows_cap, d, d_ff, dtype;
    // gathered A operand of the gate/up GEMM: row r is a[a_rows[r]] (a has
    // a_count rows); nullptr: row r is a[r]
    const int32_t* a_rows = nullptr;
    int a_count = 0;
    // stream-K split threshold in K-steps of average idle time per workgroup
    // (negative: the library default)
    int split_min_idle = -1;
    FoldArgs fold;
};
// whether launch_ffn folds the combine into the down projection for these
// arguments (bf16 256-row tiles, d a multiple of 128)
bool ffn_can_fold(const FfnArgs& a);
// counters of the folded combine: one int per (token, 128-column chunk)
inline size_t down_combine_ws_bytes(int T, int d) { return (size_t)4 * (T > 0 ? T : 1) * ((d + 127) / 128); }

// Row of the A operand that GEMM row r reads: a_rows[r] clamped into the
// source, or r itself when the operand is not gathered.
__device__ __forceinline__ int gathered_row(const int32_t* a_rows, int a_count, int r) {
    if (!a_rows) return r;
    return min(max(a_rows[r], 0), a_count - 1);
}
// bytes of the stream-K workspace on the current device
size_t ffn_workspace_bytes();
// part: 0 = both GEMMs, 1 = gate/up only, 2 = down only
hipError_t launch_ffn(const FfnArgs& a, hipStream_t s, int part = 0);
// skinny path for decode-sized batches (bf16, capacity of at most 64 rows per
// segment on average); launch_ffn takes it when ffn_skinny_fits
bool ffn_skinny_fits(const FfnArgs& a);
hipError_t launch_ffn_skinny(const FfnArgs& a, hipStream_t s, int part);

struct CombineArgs {
    const int32_t* slot_row;
    const float* slot_gate;
    const void* y;
    const void* y_shared;
    void* out;
    int T, k, d, elem_bytes;
    int64_t rows_cap;
};
hipError_t launch_combine(const CombineArgs& a, hipStream_t s);

}  // namespace bmoe
