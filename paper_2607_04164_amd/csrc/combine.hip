// Weighted sum of a token's united-expert outputs back in token order (the
// layer output of Sec. 2.1 with the per-group gate weights), plus the
// always-on shared-expert output when there is one.
// One wave per token; each lane owns 16-byte column chunks; the slot rows are
// gathered with 128-bit loads, accumulated in fp32 in slot order, and the row
// is written once with 128-bit streaming stores. When the expert-output buffer
// (its row capacity times the row size) is larger than the last-level cache
// (256 MiB) its rows are read with streaming loads too; smaller ones are often
// still cached from the down projection.
#include "bmoe_common.h"
#include "stream_io.h"

namespace bmoe {
namespace {

template <typename T>
struct Vec;
template <>
struct Vec<uint16_t> {  // 8 bf16 per chunk
    static constexpr int N = 8;
    __device__ static void load(const uint4& v, float* f) {
        const uint32_t* u = (const uint32_t*)&v;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            f[2 * i] = __uint_as_float(u[i] << 16);
            f[2 * i + 1] = __uint_as_float(u[i] & 0xffff0000u);
        }
    }
    __device__ static uint4 store(const float* f) {
        uint4 v;
        v.x = pack_bf16x2(f[0], f[1]);
        v.y = pack_bf16x2(f[2], f[3]);
        v.z = pack_bf16x2(f[4], f[5]);
        v.w = pack_bf16x2(f[6], f[7]);
        return v;
    }
};
template <>
struct Vec<float> {  // 4 floats per chunk
    static constexpr int N = 4;
    __device__ static void load(const uint4& v, float* f) {
        f[0] = __uint_as_float(v.x);
        f[1] = __uint_as_float(v.y);
        f[2] = __uint_as_float(v.z);
        f[3] = __uint_as_float(v.w);
    }
    __device__ static uint4 store(const float* f) {
        return make_uint4(__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]),
                          __float_as_uint(f[3]));
    }
};

template <typename E, int U, bool STREAM_IN>
__global__ __launch_bounds__(256) void combine_kernel(const int32_t* __restrict__ slot_row,
                                                      const float* __restrict__ slot_gate,
                                                      const uint4* __restrict__ y,
                                                      const uint4* __restrict__ y_shared,
                                                      uint4* __restrict__ out, int T, int k, int nch,
                                                      int64_t rows_cap) {
    constexpr int N = Vec<E>::N;
    const int tid = threadIdx.x, lane = tid & 63;
    const int t = blockIdx.x * 4 + (tid >> 6);
    if (t >= T) return;
    int row = -1;
    float gate = 0.f;
    if (lane < k) {
        row = slot_row[(size_t)t * k + lane];
        gate = slot_gate[(size_t)t * k + lane];
        if (row >= rows_cap) row = -1;
    }
    for (int c0 = lane; c0 < nch; c0 += 64 * U) {
        float acc[U][N];
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int j = 0; j < N; ++j) acc[u][j] = 0.f;
        for (int i = 0; i < k; ++i) {
            const int r = __shfl(row, i);
            const float g = __shfl(gate, i);
            if (r < 0) continue;
            const uint4* src = y + (size_t)r * nch;
            uint4 v[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int c = c0 + 64 * u;
                v[u] = c < nch ? (STREAM_IN ? load_stream(src + c) : src[c]) : make_uint4(0, 0, 0, 0);
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                float f[N];
                Vec<E>::load(v[u], f);
#pragma unroll
                for (int j = 0; j < N; ++j) acc[u][j] = fmaf(g, f[j], acc[u][j]);
            }
        }
        if (y_shared) {
            const uint4* src = y_shared + (size_t)t * nch;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int c = c0 + 64 * u;
                if (c < nch) {
                    float f[N];
                    Vec<E>::load(src[c], f);
#pragma unroll
                    for (int j = 0; j < N; ++j) acc[u][j] += f[j];
                }
            }
        }
        uint4* dst = out + (size_t)t * nch;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int c = c0 + 64 * u;
            if (c < nch) store_stream(dst + c, Vec<E>::store(acc[u]));
        }
    }
}

template <typename E, bool STREAM_IN>
void launch_combine_t(const CombineArgs& a, int nch, hipStream_t s) {
    hipLaunchKernelGGL((combine_kernel<E, 4, STREAM_IN>), dim3(ceil_div(a.T, 4)), dim3(256), 0, s,
                       a.slot_row, a.slot_gate, (const uint4*)a.y, (const uint4*)a.y_shared,
                       (uint4*)a.out, a.T, a.k, nch, a.rows_cap);
}

}  // namespace

hipError_t launch_combine(const CombineArgs& a, hipStream_t s) {
    if (a.T == 0) return hipSuccess;
    const int nch = a.d * a.elem_bytes / 16;
    const int64_t rows = a.rows_cap < (int64_t)a.T * a.k ? a.rows_cap : (int64_t)a.T * a.k;
    const bool stream_in = rows * a.d * a.elem_bytes >= ((int64_t)256 << 20);
    if (a.elem_bytes == 2) {
        if (stream_in) launch_combine_t<uint16_t, true>(a, nch, s);
        else launch_combine_t<uint16_t, false>(a, nch, s);
    } else {
        if (stream_in) launch_combine_t<float, true>(a, nch, s);
        else launch_combine_t<float, false>(a, nch, s);
    }
    return hipGetLastError();
}

}  // namespace bmoe
