// Group rows for the united experts: the sets G_r of the map (Eq. 2) filled
// with (token, group) pairs, in ascending token order within a group.
//
// Kernel 1 (hist_scan), one workgroup per tile of 256 tokens, tiles numbered
// by an atomic ticket in start order:
//   - each valid slot sets its token's bit in a per-group 256-bit LDS mask
//     (LDS atomic OR); popcounts give the tile's group counts and every
//     slot's stable rank inside the tile;
//   - single-pass decoupled look-back: the tile publishes its counts, walks
//     back over earlier tiles' published counts / inclusive prefixes until it
//     meets a prefix (a segment of a wave's lanes per group, reading as many
//     predecessors per step as it has lanes), then
//     publishes its own inclusive prefix;
//   - slot_row receives the row relative to the group start; the last tile
//     writes the group counts and their exclusive prefix (offsets).
// Kernel 2 (permute), one wave per token: adds offsets[group] to the relative
// row, writes perm_token, and copies x[t] into each of its rows with 128-bit
// loads and stores. Workgroup 0 clears the look-back state for the next call.
// At most 256 tokens (one tile) take a single kernel that does both.
#include <algorithm>
#include <mutex>

#include "bmoe_common.h"
#include "stream_io.h"

namespace bmoe {
namespace {

constexpr int kTile = 256;
constexpr int kMaxDevices = 64;
constexpr uint32_t kFlagAgg = 1u, kFlagPrefix = 2u;
// Upper bound on polls of one predecessor's status word. Predecessors publish
// without waiting, so the bound is only reached if the workspace was not
// zeroed before the first call; the walk then gives up instead of hanging.
constexpr int kMaxPolls = 1 << 20;

// Workspace: the tile ticket, the call's error word and one status word per
// (tile, group). A clean call finds ticket 0, so its tiles draw tickets
// 0 .. ntiles-1 and tile 0 clears the error word. A ticket at or past ntiles
// (the workspace was not zero) or a look-back that gives up sets the error
// word; the permute kernel then writes the "no rows" result (counts 0,
// offsets 0 with offsets[G] = -1, every slot_row -1) and nothing else, and
// its last workgroup to finish (counted in `done`) clears the error word. The
// permute kernel's workgroup 0 clears the ticket and the status words, so the
// next call starts clean either way.
struct DispatchWs {
    int32_t ticket;
    int32_t err;
    int32_t done;
    int32_t pad[61];
    // followed by uint64_t status[ntiles * G]
};

__device__ __forceinline__ uint64_t pack_status(uint32_t flag, uint32_t value) {
    return ((uint64_t)flag << 32) | value;
}

__global__ __launch_bounds__(kTile) void hist_scan_kernel(const int32_t* __restrict__ slot_group,
                                                          int32_t* __restrict__ slot_row,
                                                          int32_t* __restrict__ counts,
                                                          int32_t* __restrict__ offsets, void* ws,
                                                          int T, int k, int G, int ntiles) {
    __shared__ unsigned long long masks[BMOE_MAX_EXPERTS][kTile / 64];
    __shared__ int s_tile;
    __shared__ int s_excl[BMOE_MAX_EXPERTS];
    __shared__ int s_cnt[BMOE_MAX_EXPERTS];
    __shared__ int s_scan[256];
    DispatchWs* hdr = (DispatchWs*)ws;
    uint64_t* status = (uint64_t*)((char*)ws + sizeof(DispatchWs));
    const int tid = threadIdx.x;

    if (tid == 0) s_tile = atomicAdd(&hdr->ticket, 1);
    for (int g = tid; g < G; g += kTile) {
#pragma unroll
        for (int w = 0; w < kTile / 64; ++w) masks[g][w] = 0ull;
    }
    __syncthreads();
    const int tile = s_tile;
    if (tile >= ntiles) {
        // the workspace was not zero: no out-of-range writes, the call reports it
        if (tid == 0) __hip_atomic_store(&hdr->err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return;
    }
    if (tile == 0 && tid == 0) __hip_atomic_store(&hdr->err, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int t = tile * kTile + tid;
    const bool tok = t < T;

    int grp[BMOE_MAX_TOPK];
#pragma unroll
    for (int i = 0; i < BMOE_MAX_TOPK; ++i) {
        grp[i] = -1;
        if (i < k && tok) {
            int g = slot_group[(size_t)t * k + i];
            if (g >= 0 && g < G) {
                grp[i] = g;
                atomicOr(&masks[g][tid >> 6], 1ull << (tid & 63));
            }
        }
    }
    __syncthreads();

    if (tid < G) {
        int c = 0;
#pragma unroll
        for (int w = 0; w < kTile / 64; ++w) c += __popcll(masks[tid][w]);
        s_cnt[tid] = c;
        __hip_atomic_store(status + (size_t)tile * G + tid,
                           pack_status(tile == 0 ? kFlagPrefix : kFlagAgg, (uint32_t)c),
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();

    // Look-back. Each wave takes gpw groups (a power of two, 4 * gpw >= G) and
    // gives each a segment of lpg = 64 / gpw lanes; lane i of a segment reads
    // the status of tile j0 - i, so one round trip covers lpg predecessors of
    // every group of the wave. Every earlier tile took its ticket before this
    // one and publishes its counts without waiting on anything, so each window
    // fills and the walk terminates. A status word holds both its flag and its
    // count and nothing else is published through it, so relaxed device-scope
    // atomics suffice (acquire/release would add an L2 invalidate or write-back
    // to every poll and publish).
    {
        const int wave = tid >> 6, lane = tid & 63;
        int gpw = 1;
        while (gpw * (kTile / 64) < G) gpw <<= 1;
        const int lpg = 64 / gpw;
        const int sl = lane & (lpg - 1), sb = lane - sl;
        const uint64_t segmask = lpg == 64 ? ~0ull : ((1ull << lpg) - 1ull);
        const int g = wave * gpw + lane / lpg;
        const bool gv = g < G;
        const int c = gv ? s_cnt[g] : 0;
        int excl = 0, j0 = tile - 1, polls = 0;
        bool done = !gv || j0 < 0;
        while (__ballot(!done) != 0ull) {
            const int j = j0 - sl;
            uint64_t sv = pack_status(kFlagPrefix, 0u);
            if (!done && j >= 0)
                sv = __hip_atomic_load(status + (size_t)j * G + g, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
            const uint32_t flag = (uint32_t)(sv >> 32);
            const uint64_t pm = (__ballot(flag == kFlagPrefix) >> sb) & segmask;
            const uint64_t zm = (__ballot(flag == 0u) >> sb) & segmask;
            const int np = pm ? __ffsll((unsigned long long)pm) - 1 : lpg;  // nearest prefix
            const uint64_t need = np >= lpg ? segmask : ((2ull << np) - 1ull);
            const bool wait = !done && (zm & need) != 0ull;
            int v = (!done && !wait && sl <= np) ? (int)(uint32_t)sv : 0;
            for (int m = lpg >> 1; m >= 1; m >>= 1) v += __shfl_xor(v, m);
            if (!done && !wait) {
                excl += v;
                if (np < lpg) done = true;
                else j0 -= lpg;
            }
            if (__ballot(wait) != 0ull) {
                if (++polls > kMaxPolls) {  // workspace was not zeroed: the call reports it
                    if (lane == 0) __hip_atomic_store(&hdr->err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    break;
                }
                __builtin_amdgcn_s_sleep(1);
            }
        }
        if (gv && sl == 0) {
            if (tile > 0)
                __hip_atomic_store(status + (size_t)tile * G + g,
                                   pack_status(kFlagPrefix, (uint32_t)(excl + c)), __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
            s_excl[g] = excl;
        }
    }
    __syncthreads();

    if (tok) {
        const int w = tid >> 6;
        const unsigned long long lt = (1ull << (tid & 63)) - 1ull;
#pragma unroll
        for (int i = 0; i < BMOE_MAX_TOPK; ++i) {
            if (i < k) {
                int rel = -1;
                const int g = grp[i];
                if (g >= 0) {
                    int rank = __popcll(masks[g][w] & lt);
                    for (int ww = 0; ww < w; ++ww) rank += __popcll(masks[g][ww]);
                    rel = s_excl[g] + rank;
                }
                slot_row[(size_t)t * k + i] = rel;
            }
        }
    }

    if (tile == ntiles - 1) {
        const int total = tid < G ? s_excl[tid] + s_cnt[tid] : 0;
        int sum;
        const int ex = block_exclusive_scan_256(total, s_scan, &sum);
        if (tid < G) {
            counts[tid] = total;
            offsets[tid] = ex;
        }
        if (tid == 0) offsets[G] = sum;
    }
}

// First step of both permute kernels. Workgroup 0 leaves the look-back state
// (ticket and status words) all zero for the next call; nothing in this
// kernel reads it. When the histogram kernel reported an error, the call's
// result is "no rows": workgroup 0 writes counts 0 and offsets 0 with
// offsets[G] = -1, every thread sets its n_slots slots (from slot index o0)
// to -1, and the kernel stops (returns true).
__device__ __forceinline__ bool permute_prologue(void* ws, int32_t* slot_row, int32_t* counts, int32_t* offsets,
                                                 int T, int k, int G, int ntiles, int64_t o0, int n_slots) {
    DispatchWs* hdr = (DispatchWs*)ws;
    const int tid = threadIdx.x;
    const int err = __hip_atomic_load(&hdr->err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (blockIdx.x == 0) {
        uint64_t* status = (uint64_t*)((char*)ws + sizeof(DispatchWs));
        const int n = ntiles * G;
        for (int i = tid; i < n; i += 256) status[i] = 0ull;
        if (tid == 0) hdr->ticket = 0;
        if (err) {
            for (int g = tid; g <= G; g += 256) {
                if (g < G) counts[g] = 0;
                offsets[g] = g < G ? 0 : -1;
            }
        }
    }
    if (!err) return false;
    for (int i = 0; i < n_slots; ++i)
        if (o0 + i < (int64_t)T * k) slot_row[o0 + i] = -1;
    // every workgroup has read the error word (err is the same for all of
    // them: nothing clears it before the last one is counted)
    __syncthreads();
    if (tid == 0) {
        __threadfence();
        if (atomicAdd(&hdr->done, 1) == (int)gridDim.x - 1) {
            __hip_atomic_store(&hdr->err, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(&hdr->done, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
    return true;
}

// Clears a dispatch workspace of `bytes` bytes (a multiple of 8).
__global__ __launch_bounds__(256) void ws_clear_kernel(uint64_t* ws, int64_t n_words) {
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n_words; i += (int64_t)gridDim.x * 256)
        ws[i] = 0ull;
}

// One wave per token. VEC: 16-byte chunks each lane moves per batch.
template <int VEC>
__global__ __launch_bounds__(256) void permute_kernel(const int32_t* __restrict__ slot_group,
                                                      int32_t* __restrict__ slot_row,
                                                      int32_t* __restrict__ counts,
                                                      int32_t* __restrict__ offsets,
                                                      int32_t* __restrict__ perm_token,
                                                      const uint4* __restrict__ x,
                                                      uint4* __restrict__ x_perm, void* ws, int T,
                                                      int k, int G, int nch, int ntiles, int rows_cap) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int t = blockIdx.x * 4 + (tid >> 6);
    if (permute_prologue(ws, slot_row, counts, offsets, T, k, G, ntiles, (int64_t)t * k + lane, lane < k ? 1 : 0))
        return;
    if (t >= T) return;
    int row = -1;
    if (lane < k) {
        const size_t o = (size_t)t * k + lane;
        const int g = slot_group[o];
        if (g >= 0 && g < G) {
            row = offsets[g] + slot_row[o];
            if (row < 0 || row >= rows_cap) row = -1;
            else perm_token[row] = t;
        }
        slot_row[o] = row;
    }
    const uint4* src = x + (size_t)t * nch;
    int rows[BMOE_MAX_TOPK];
#pragma unroll
    for (int i = 0; i < BMOE_MAX_TOPK; ++i) rows[i] = i < k ? __shfl(row, i) : -1;
    for (int c0 = lane; c0 < nch; c0 += 64 * VEC) {
        uint4 v[VEC];
#pragma unroll
        for (int u = 0; u < VEC; ++u) {
            const int c = c0 + 64 * u;
            v[u] = src[c < nch ? c : 0];
        }
#pragma unroll
        for (int i = 0; i < BMOE_MAX_TOPK; ++i) {
            if (rows[i] >= 0) {
                uint4* dst = x_perm + (size_t)rows[i] * nch;
#pragma unroll
                for (int u = 0; u < VEC; ++u) {
                    const int c = c0 + 64 * u;
                    if (c < nch) store_stream(dst + c, v[u]);
                }
            }
        }
    }
}

// The permutation without the row copies (for an FFN that gathers its rows
// from x itself): one thread per slot writes its row and the row's token.
__global__ __launch_bounds__(256) void permute_index_kernel(const int32_t* __restrict__ slot_group,
                                                            int32_t* __restrict__ slot_row,
                                                            int32_t* __restrict__ counts,
                                                            int32_t* __restrict__ offsets,
                                                            int32_t* __restrict__ perm_token, void* ws, int T,
                                                            int k, int G, int ntiles, int rows_cap) {
    const int tid = threadIdx.x;
    const int64_t o = (int64_t)blockIdx.x * 256 + tid;
    if (permute_prologue(ws, slot_row, counts, offsets, T, k, G, ntiles, o, 1)) return;
    if (o >= (int64_t)T * k) return;
    const int g = slot_group[o];
    int row = -1;
    if (g >= 0 && g < G) {
        row = offsets[g] + slot_row[o];
        if (row < 0 || row >= rows_cap) row = -1;
        else perm_token[row] = (int)(o / k);
    }
    slot_row[o] = row;
}

// Dispatch of at most one tile of tokens (T <= 256) in one kernel: every
// workgroup rebuilds the tile's per-group token masks and their prefix in
// LDS (a few hundred slots), so no workgroup waits on another and the
// histogram kernel's launch is saved; workgroup w then takes tokens
// 4w .. 4w+3, one wave each, as the permute kernel does. The workspace is
// only read: a ticket left set by a call cut short gives the "no rows"
// result of the two-kernel path, and the last workgroup to finish (counted
// in `done`, after every workgroup has read the ticket) clears it.
template <int VEC>
__global__ __launch_bounds__(256) void dispatch_small_kernel(const int32_t* __restrict__ slot_group,
                                                             int32_t* __restrict__ slot_row,
                                                             int32_t* __restrict__ counts,
                                                             int32_t* __restrict__ offsets,
                                                             int32_t* __restrict__ perm_token,
                                                             const uint4* __restrict__ x, uint4* __restrict__ x_perm,
                                                             void* ws, int T, int k, int G, int nch, int rows_cap) {
    __shared__ unsigned long long masks[BMOE_MAX_EXPERTS][kTile / 64];
    __shared__ int s_off[BMOE_MAX_EXPERTS];
    __shared__ int s_scan[256];
    DispatchWs* hdr = (DispatchWs*)ws;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int t = blockIdx.x * 4 + wave;  // this wave's token
    const bool stale = __hip_atomic_load(&hdr->ticket, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0;
    if (stale) {
        if (blockIdx.x == 0) {
            for (int g = tid; g <= G; g += 256) {
                if (g < G) counts[g] = 0;
                offsets[g] = g < G ? 0 : -1;
            }
        }
        if (t < T && lane < k) slot_row[(size_t)t * k + lane] = -1;
        __syncthreads();  // every wave of this workgroup has read the ticket
        if (tid == 0) {
            __threadfence();
            if (atomicAdd(&hdr->done, 1) == (int)gridDim.x - 1) {
                uint64_t* status = (uint64_t*)((char*)ws + sizeof(DispatchWs));
                for (int g = 0; g < G; ++g) status[g] = 0ull;
                __hip_atomic_store(&hdr->ticket, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(&hdr->err, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(&hdr->done, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
        return;
    }
    for (int g = tid; g < G; g += 256) {
#pragma unroll
        for (int w = 0; w < kTile / 64; ++w) masks[g][w] = 0ull;
    }
    __syncthreads();
    // thread tid sets the bit of token tid in the mask of each of its groups
    if (tid < T) {
        for (int i = 0; i < k; ++i) {
            const int g = slot_group[(size_t)tid * k + i];
            if (g >= 0 && g < G) atomicOr(&masks[g][tid >> 6], 1ull << (tid & 63));
        }
    }
    __syncthreads();
    int c = 0;
    if (tid < G) {
#pragma unroll
        for (int w = 0; w < kTile / 64; ++w) c += __popcll(masks[tid][w]);
    }
    int sum;
    const int ex = block_exclusive_scan_256(c, s_scan, &sum);
    if (tid < G) {
        s_off[tid] = ex;
        if (blockIdx.x == 0) {
            counts[tid] = c;
            offsets[tid] = ex;
        }
    }
    if (blockIdx.x == 0 && tid == 0) offsets[G] = sum;
    __syncthreads();
    if (t >= T) return;
    int row = -1;
    if (lane < k) {
        const size_t o = (size_t)t * k + lane;
        const int g = slot_group[o];
        if (g >= 0 && g < G) {
            const int w = t >> 6;
            int rank = __popcll(masks[g][w] & ((1ull << (t & 63)) - 1ull));
            for (int ww = 0; ww < w; ++ww) rank += __popcll(masks[g][ww]);
            row = s_off[g] + rank;
            if (row < 0 || row >= rows_cap) row = -1;
            else perm_token[row] = t;
        }
        slot_row[o] = row;
    }
    if (x_perm == nullptr) return;
    const uint4* src = x + (size_t)t * nch;
    int rows[BMOE_MAX_TOPK];
#pragma unroll
    for (int i = 0; i < BMOE_MAX_TOPK; ++i) rows[i] = i < k ? __shfl(row, i) : -1;
    for (int c0 = lane; c0 < nch; c0 += 64 * VEC) {
        uint4 v[VEC];
#pragma unroll
        for (int u = 0; u < VEC; ++u) {
            const int cc = c0 + 64 * u;
            v[u] = src[cc < nch ? cc : 0];
        }
#pragma unroll
        for (int i = 0; i < BMOE_MAX_TOPK; ++i) {
            if (rows[i] >= 0) {
                uint4* dst = x_perm + (size_t)rows[i] * nch;
#pragma unroll
                for (int u = 0; u < VEC; ++u) {
                    const int cc = c0 + 64 * u;
                    if (cc < nch) store_stream(dst + cc, v[u]);
                }
            }
        }
    }
}

}  // namespace

size_t dispatch_ws_bytes(int T, int G) {
    const size_t ntiles = (size_t)ceil_div(T > 0 ? T : 1, kTile);
    return sizeof(DispatchWs) + ntiles * (size_t)G * sizeof(uint64_t);
}

static hipError_t clear_ws(void* ws, size_t bytes, hipStream_t s) {
    const int64_t words = (int64_t)(bytes / 8);
    const int64_t blocks = std::min<int64_t>((words + 255) / 256, 256);
    hipLaunchKernelGGL(ws_clear_kernel, dim3((unsigned)blocks), dim3(256), 0, s, (uint64_t*)ws, words);
    return hipGetLastError();
}

hipError_t launch_dispatch(const DispatchArgs& a, hipStream_t s) {
    if (a.T == 0) return hipSuccess;
    if (a.T <= kTile) {
        // one tile: a single kernel (no look-back, no second launch)
        const int nch = a.x_perm ? a.d * a.elem_bytes / 16 : 0;
        if (nch > 256)
            hipLaunchKernelGGL(dispatch_small_kernel<8>, dim3(ceil_div(a.T, 4)), dim3(256), 0, s, a.slot_group,
                               a.slot_row, a.counts, a.offsets, a.perm_token, (const uint4*)a.x,
                               (uint4*)a.x_perm, a.ws, a.T, a.k, a.G, nch, a.T * a.k);
        else
            hipLaunchKernelGGL(dispatch_small_kernel<4>, dim3(ceil_div(a.T, 4)), dim3(256), 0, s, a.slot_group,
                               a.slot_row, a.counts, a.offsets, a.perm_token, (const uint4*)a.x,
                               (uint4*)a.x_perm, a.ws, a.T, a.k, a.G, nch, a.T * a.k);
        return hipGetLastError();
    }
    const int ntiles = ceil_div(a.T, kTile);
    hipLaunchKernelGGL(hist_scan_kernel, dim3(ntiles), dim3(kTile), 0, s, a.slot_group, a.slot_row,
                       a.counts, a.offsets, a.ws, a.T, a.k, a.G, ntiles);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (a.x_perm == nullptr) {
        const int64_t slots = (int64_t)a.T * a.k;
        hipLaunchKernelGGL(permute_index_kernel, dim3((unsigned)((slots + 255) / 256)), dim3(256), 0, s,
                           a.slot_group, a.slot_row, a.counts, a.offsets, a.perm_token, a.ws, a.T, a.k, a.G,
                           ntiles, a.T * a.k);
    } else {
        const int nch = a.d * a.elem_bytes / 16;
        // a row of up to 8 KB in one batch of loads per lane
        if (nch > 256)
            hipLaunchKernelGGL(permute_kernel<8>, dim3(ceil_div(a.T, 4)), dim3(256), 0, s, a.slot_group,
                               a.slot_row, a.counts, a.offsets, a.perm_token, (const uint4*)a.x,
                               (uint4*)a.x_perm, a.ws, a.T, a.k, a.G, nch, ntiles, a.T * a.k);
        else
            hipLaunchKernelGGL(permute_kernel<4>, dim3(ceil_div(a.T, 4)), dim3(256), 0, s, a.slot_group,
                               a.slot_row, a.counts, a.offsets, a.perm_token, (const uint4*)a.x,
                               (uint4*)a.x_perm, a.ws, a.T, a.k, a.G, nch, ntiles, a.T * a.k);
    }
    e = hipGetLastError();
    // the histogram kernel ran but its partner did not: leave the workspace
    // zero for the next call (if this launch fails too, the next call's
    // histogram sees the stale ticket and reports it)
    if (e != hipSuccess) (void)clear_ws(a.ws, dispatch_ws_bytes(a.T, a.G), s);
    return e;
}

// ---- the allocation-free variant: the workspace is a device array of the
// library itself (one copy per GPU, found through hipGetSymbolAddress once
// per device and kept; never passed by its host-side name)

static __device__ __align__(256) uint64_t scratch[BMOE_DISPATCH_SCRATCH_BYTES / 8];

static std::mutex g_scratch_mu;
static void* g_scratch_ptr[kMaxDevices];

static hipError_t scratch_address(void** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[dev] == nullptr) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (p == nullptr) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

hipError_t launch_dispatch_noalloc(const DispatchArgs& a0, hipStream_t s) {
    if (a0.T == 0) return hipSuccess;
    const size_t bytes = dispatch_ws_bytes(a0.T, a0.G);
    if (bytes > (size_t)BMOE_DISPATCH_SCRATCH_BYTES) return hipErrorInvalidValue;  // checked by the caller
    DispatchArgs a = a0;
    hipError_t e = scratch_address(&a.ws);
    if (e != hipSuccess) return e;
    // every call starts from a cleared array (by a kernel, not a memset, so
    // the call may be captured into a graph)
    e = clear_ws(a.ws, bytes, s);
    if (e != hipSuccess) return e;
    return launch_dispatch(a, s);
}

}  // namespace bmoe
