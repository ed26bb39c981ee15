// Streaming 128-bit loads and stores for the HBM-bound row kernels (permute,
// combine) of libbrownout_moe (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bmoe {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Streaming 128-bit store and load (nontemporal hint): for rows that one
// kernel writes or reads exactly once, so they do not displace reused lines.
__device__ __forceinline__ void store_stream(uint4* p, const uint4& v) {
    __builtin_nontemporal_store(__builtin_bit_cast(u32x4, v), (u32x4*)p);
}
__device__ __forceinline__ uint4 load_stream(const uint4* p) {
    return __builtin_bit_cast(uint4, __builtin_nontemporal_load((const u32x4*)p));
}

}  // namespace bmoe
