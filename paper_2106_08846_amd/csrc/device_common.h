// Small device/host helpers shared by libbsr's kernels.
#pragma once

#include <hip/hip_runtime.h>

#include "bsr_internal.h"

namespace bsr {

inline hipStream_t as_stream(void *s) { return reinterpret_cast<hipStream_t>(s); }

// Status of the launch just enqueued (records the HIP error text on failure).
inline bsr_status launch_status() {
    hipError_t e = hipGetLastError();
    if (e == hipSuccess) return BSR_OK;
    set_last_hip_error(hipGetErrorString(e));
    return BSR_ERR_HIP;
}

__device__ __forceinline__ int64_t clamp64(int64_t v, int64_t lo, int64_t hi) {
    return v < lo ? lo : (v > hi ? hi : v);
}

__device__ __forceinline__ int clampi(int v, int lo, int hi) {
    return v < lo ? lo : (v > hi ? hi : v);
}

// bf16 bit pattern -> fp32 value (exact widening).
__device__ __forceinline__ float bf16_bits_to_float(unsigned short h) {
    return __uint_as_float(static_cast<unsigned int>(h) << 16);
}

// Grid size for a grid-stride loop over `n` items with `threads` per block.
inline unsigned grid_for(int64_t n, int threads, int64_t cap = int64_t(1) << 20) {
    int64_t g = (n + threads - 1) / threads;
    if (g < 1) g = 1;
    if (g > cap) g = cap;
    return static_cast<unsigned>(g);
}

}  // namespace bsr
