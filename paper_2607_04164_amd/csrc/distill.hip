// Grouping-search kernels of one layer (Sec. 4.3): the parameter-average
// initialisation of the united experts, and the distillation error of every
// group against its routing-weighted target (Eq. 5) with the
// routing-frequency-weighted total (Eq. 3, Eq. 6).
//
// Both are bound by HBM bandwidth. united_init streams every expert weight
// once and writes every united weight once: one thread per 16-byte chunk of a
// united matrix sums that chunk of its members (ascending expert index) and
// divides by the member count. distill_mse streams the member experts'
// outputs and the united experts' outputs once: a workgroup owns a range of
// calibration tokens of one group, each thread forms the target of a 16-byte
// chunk in fp32 (Eq. 5, alphas from the frequencies) and accumulates the
// squared difference in fp64; workgroup sums go to a workspace in a fixed
// slot, and a one-workgroup pass adds them in slot order, so results do not
// depend on scheduling.
#include "bmoe_common.h"

namespace bmoe {
namespace {

constexpr int kDThreads = 256;

// Members of group r (ascending expert index) into s_mem; returns the count.
// Every thread of the (256-thread) workgroup must call it.
__device__ __forceinline__ int group_members(const int32_t* e2g, int E, int r, int* s_mem, int* s_scan) {
    const int tid = threadIdx.x;
    const bool in = tid < E && e2g[tid] == r;
    int n;
    const int pos = block_exclusive_scan_256(in ? 1 : 0, s_scan, &n);
    if (in) s_mem[pos] = tid;
    __syncthreads();
    return n;
}

template <typename V>
__device__ __forceinline__ void load_chunk(const V* p, float (&v)[16 / sizeof(V)]);
template <>
__device__ __forceinline__ void load_chunk<uint16_t>(const uint16_t* p, float (&v)[8]) {
    const uint4 q = *(const uint4*)p;
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        v[2 * i] = __uint_as_float(w[i] << 16);
        v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
}
template <>
__device__ __forceinline__ void load_chunk<float>(const float* p, float (&v)[4]) {
    const float4 q = *(const float4*)p;
    v[0] = q.x;
    v[1] = q.y;
    v[2] = q.z;
    v[3] = q.w;
}

// dst[r] = (sum of src[e] over the members e of group r) / count, per element;
// blockIdx.y = r, blockIdx.z = matrix (gate, up, down). Empty groups get zeros.
template <typename V>
__global__ __launch_bounds__(kDThreads) void united_init_kernel(const int32_t* __restrict__ e2g, int E,
                                                                const V* __restrict__ s0, const V* __restrict__ s1,
                                                                const V* __restrict__ s2, V* __restrict__ d0,
                                                                V* __restrict__ d1, V* __restrict__ d2,
                                                                int64_t nchunk) {
    constexpr int EPC = 16 / sizeof(V);
    __shared__ int s_mem[BMOE_MAX_EXPERTS];
    __shared__ int s_scan[256];
    const int r = blockIdx.y, mat = blockIdx.z;
    const int n = group_members(e2g, E, r, s_mem, s_scan);
    const V* src = mat == 0 ? s0 : mat == 1 ? s1 : s2;
    V* dst = mat == 0 ? d0 : mat == 1 ? d1 : d2;
    const int64_t per = nchunk * EPC;  // elements per matrix
    for (int64_t c = (int64_t)blockIdx.x * kDThreads + threadIdx.x; c < nchunk;
         c += (int64_t)gridDim.x * kDThreads) {
        if constexpr (sizeof(V) == 2) {
            float acc[EPC];
#pragma unroll
            for (int i = 0; i < EPC; ++i) acc[i] = 0.f;
            for (int m = 0; m < n; ++m) {
                float v[EPC];
                load_chunk<V>(src + (size_t)s_mem[m] * per + c * EPC, v);
#pragma unroll
                for (int i = 0; i < EPC; ++i) acc[i] += v[i];
            }
            uint32_t o[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float a = n ? acc[2 * i] / (float)n : 0.f, b = n ? acc[2 * i + 1] / (float)n : 0.f;
                o[i] = (uint32_t)f32_to_bf16(a) | ((uint32_t)f32_to_bf16(b) << 16);
            }
            *(uint4*)(dst + (size_t)r * per + c * EPC) = make_uint4(o[0], o[1], o[2], o[3]);
        } else {
            double acc[EPC];
#pragma unroll
            for (int i = 0; i < EPC; ++i) acc[i] = 0.0;
            for (int m = 0; m < n; ++m) {
                float v[EPC];
                load_chunk<V>(src + (size_t)s_mem[m] * per + c * EPC, v);
#pragma unroll
                for (int i = 0; i < EPC; ++i) acc[i] += (double)v[i];
            }
            float4 o;
            o.x = n ? (float)(acc[0] / n) : 0.f;
            o.y = n ? (float)(acc[1] / n) : 0.f;
            o.z = n ? (float)(acc[2] / n) : 0.f;
            o.w = n ? (float)(acc[3] / n) : 0.f;
            *(float4*)(dst + (size_t)r * per + c * EPC) = o;
        }
    }
}

// Alphas of Eq. 5 for the members of one group (equal weights when the
// members' frequencies sum to zero), into s_alpha; every thread calls it.
__device__ __forceinline__ void group_alphas(const float* w, const int* s_mem, int n, float* s_alpha) {
    if (threadIdx.x == 0) {
        double tot = 0.0;
        for (int m = 0; m < n; ++m) tot += (double)w[s_mem[m]];
        for (int m = 0; m < n; ++m) s_alpha[m] = tot > 0.0 ? (float)((double)w[s_mem[m]] / tot) : 1.f / (float)n;
    }
    __syncthreads();
}

// Partial sums of (u - t)^2 over tokens [t0, t1) of group r = blockIdx.y.
template <typename V>
__global__ __launch_bounds__(kDThreads) void distill_partial_kernel(const int32_t* __restrict__ e2g, int E,
                                                                    const float* __restrict__ w,
                                                                    const V* __restrict__ y_e,
                                                                    const V* __restrict__ y_u, int T, int d,
                                                                    double* __restrict__ part) {
    constexpr int EPC = 16 / sizeof(V);
    __shared__ int s_mem[BMOE_MAX_EXPERTS];
    __shared__ int s_scan[256];
    __shared__ float s_alpha[BMOE_MAX_EXPERTS];
    __shared__ double s_red[kDThreads];
    const int r = blockIdx.y, nb = gridDim.x, b = blockIdx.x;
    const int n = group_members(e2g, E, r, s_mem, s_scan);
    group_alphas(w, s_mem, n, s_alpha);
    const int nch = d / EPC;
    const int t0 = (int)((int64_t)T * b / nb), t1 = (int)((int64_t)T * (b + 1) / nb);
    const int nc = (t1 - t0) * nch;  // chunks of this workgroup (the host bounds T d / nb)
    double acc = 0.0;
    if (n > 0) {
        // two chunks per thread and step, every load of both issued before any
        // is used; squares added in chunk order
        constexpr int U = 2;
        for (int c0 = threadIdx.x; c0 < nc; c0 += U * kDThreads) {
            float tv[U][EPC], u[U][EPC];
#pragma unroll
            for (int q = 0; q < U; ++q)
#pragma unroll
                for (int i = 0; i < EPC; ++i) tv[q][i] = 0.f;
            bool ok[U];
            int t[U], j[U];
#pragma unroll
            for (int q = 0; q < U; ++q) {
                const int c = c0 + q * kDThreads;
                ok[q] = c < nc;
                const int cc = ok[q] ? c : 0;
                t[q] = t0 + cc / nch;
                j[q] = cc % nch;
            }
            for (int m = 0; m < n; ++m) {
                float v[U][EPC];
#pragma unroll
                for (int q = 0; q < U; ++q)
                    load_chunk<V>(y_e + ((size_t)s_mem[m] * T + t[q]) * d + (size_t)j[q] * EPC, v[q]);
                const float a = s_alpha[m];
#pragma unroll
                for (int q = 0; q < U; ++q)
#pragma unroll
                    for (int i = 0; i < EPC; ++i) tv[q][i] = fmaf(a, v[q][i], tv[q][i]);
            }
#pragma unroll
            for (int q = 0; q < U; ++q) load_chunk<V>(y_u + ((size_t)r * T + t[q]) * d + (size_t)j[q] * EPC, u[q]);
#pragma unroll
            for (int q = 0; q < U; ++q) {
                if (!ok[q]) continue;
#pragma unroll
                for (int i = 0; i < EPC; ++i) {
                    const double df = (double)(u[q][i] - tv[q][i]);
                    acc = fma(df, df, acc);
                }
            }
        }
    }
    // fixed-order tree over the workgroup
    s_red[threadIdx.x] = acc;
    __syncthreads();
    for (int off = kDThreads / 2; off > 0; off >>= 1) {
        if ((int)threadIdx.x < off) s_red[threadIdx.x] += s_red[threadIdx.x + off];
        __syncthreads();
    }
    if (threadIdx.x == 0) part[(size_t)r * nb + b] = s_red[0];
}

// mse[r] = (sum of group r's partials in slot order) / (T d); total = sum of
// beta_r mse[r] in ascending r (beta_r: the members' frequency sum).
__global__ __launch_bounds__(kDThreads) void distill_final_kernel(const int32_t* __restrict__ e2g, int E, int G,
                                                                  const float* __restrict__ w,
                                                                  const double* __restrict__ part, int nb, int T,
                                                                  int d, double* __restrict__ mse,
                                                                  double* __restrict__ total) {
    __shared__ double s_wm[BMOE_MAX_EXPERTS];  // beta_r * mse_r
    const int r = threadIdx.x;
    if (r < G) {
        double s = 0.0, beta = 0.0;
        int n = 0;
        for (int b = 0; b < nb; ++b) s += part[(size_t)r * nb + b];
        for (int e = 0; e < E; ++e)
            if (e2g[e] == r) {
                beta += (double)w[e];
                ++n;
            }
        const double m = n ? s / ((double)T * (double)d) : 0.0;
        mse[r] = m;
        s_wm[r] = beta * m;
    }
    __syncthreads();
    if (r == 0 && total) {
        double tot = 0.0;
        for (int g = 0; g < G; ++g) tot += s_wm[g];
        *total = tot;
    }
}

}  // namespace

int distill_blocks(int G, int T) {
    // about four workgroups per CU (measured: 512 or 2048 in all were slower),
    // at most one per token
    int nb = (1024 + G - 1) / G;
    return nb < T ? nb : T;
}

hipError_t launch_united_init(const UnitedInitArgs& a, hipStream_t s) {
    const int64_t elems_gu = (int64_t)a.d_ff * a.d;  // gate/up and down hold the same count
    const int epc = a.dtype == BMOE_BF16 ? 8 : 4;
    const int64_t nchunk = elems_gu / epc;
    const int64_t want = (nchunk + kDThreads - 1) / kDThreads;
    const unsigned gx = (unsigned)(want < 1024 ? want : 1024);
    dim3 grid(gx, (unsigned)a.G, 3);
    if (a.dtype == BMOE_BF16)
        hipLaunchKernelGGL(united_init_kernel<uint16_t>, grid, dim3(kDThreads), 0, s, a.e2g, a.E,
                           (const uint16_t*)a.src[0], (const uint16_t*)a.src[1], (const uint16_t*)a.src[2],
                           (uint16_t*)a.dst[0], (uint16_t*)a.dst[1], (uint16_t*)a.dst[2], nchunk);
    else
        hipLaunchKernelGGL(united_init_kernel<float>, grid, dim3(kDThreads), 0, s, a.e2g, a.E,
                           (const float*)a.src[0], (const float*)a.src[1], (const float*)a.src[2],
                           (float*)a.dst[0], (float*)a.dst[1], (float*)a.dst[2], nchunk);
    return hipGetLastError();
}

hipError_t launch_distill_mse(const DistillArgs& a, hipStream_t s) {
    const int nb = distill_blocks(a.G, a.T);
    double* part = (double*)a.ws;
    dim3 grid((unsigned)nb, (unsigned)a.G);
    if (a.dtype == BMOE_BF16)
        hipLaunchKernelGGL(distill_partial_kernel<uint16_t>, grid, dim3(kDThreads), 0, s, a.e2g, a.E, a.w,
                           (const uint16_t*)a.y_expert, (const uint16_t*)a.y_united, a.T, a.d, part);
    else
        hipLaunchKernelGGL(distill_partial_kernel<float>, grid, dim3(kDThreads), 0, s, a.e2g, a.E, a.w,
                           (const float*)a.y_expert, (const float*)a.y_united, a.T, a.d, part);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(distill_final_kernel, dim3(1), dim3(kDThreads), 0, s, a.e2g, a.E, a.G, a.w, part, nb, a.T,
                       a.d, a.mse, a.total);
    return hipGetLastError();
}

}  // namespace bmoe
