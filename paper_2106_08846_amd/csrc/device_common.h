// Small device/host helpers shared by libbsr's kernels.
#pragma once

#include <hip/hip_ext.h>
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

// Launch `kernel`, through hipExtLaunchKernel when an event pair is given so that the events
// mark the kernel's own start and end on the device.
template <typename... Params, typename... Args>
inline void launch_kernel(void (*kernel)(Params...), dim3 grid, dim3 block, size_t lds,
                          hipStream_t st, const LaunchEvents &ev, Args... args) {
    if (ev.start != nullptr || ev.stop != nullptr)
        hipExtLaunchKernelGGL(kernel, grid, block, static_cast<uint32_t>(lds), st,
                              static_cast<hipEvent_t>(ev.start),
                              static_cast<hipEvent_t>(ev.stop), 0u, static_cast<Params>(args)...);
    else
        hipLaunchKernelGGL(kernel, grid, block, static_cast<uint32_t>(lds), st,
                           static_cast<Params>(args)...);
}

__device__ __forceinline__ int64_t clamp64(int64_t v, int64_t lo, int64_t hi) {
    return v < lo ? lo : (v > hi ? hi : v);
}

__device__ __forceinline__ int clampi(int v, int lo, int hi) {
    return v < lo ? lo : (v > hi ? hi : v);
}

// A value the compiler may treat as uniform across the wave (lane 0's copy).
__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

// Raw buffer resource over [base, base + bytes): loads past the end return 0 and stores past
// it are dropped.  Word 3 is the default raw-buffer configuration for gfx9-family chips.  The
// launch plans keep every range below 2^31 bytes.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void *base, unsigned bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, int(bytes), 0x00020000);
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
