// libbsr C entry points: validate on the host, check the device, enqueue kernels.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdio>
#include <cstring>
#include <mutex>

#include "bsr_internal.h"
#include "spmm_tiled.h"

namespace bsr {

namespace {

constexpr int kMaxDevices = 64;

struct DeviceInfo {
    std::atomic<int> state{0};  // 0 unknown, 1 gfx950, -1 other architecture
    int cu_count = 0;
    size_t lds_per_block = 0;
};

DeviceInfo g_devices[kMaxDevices];
std::mutex g_device_mutex;
thread_local char g_last_hip_error[256] = "";

int current_device() {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return -1;
    return dev;
}

}  // namespace

void set_last_hip_error(const char *msg) {
    std::snprintf(g_last_hip_error, sizeof(g_last_hip_error), "%s", msg ? msg : "");
}

bsr_status ensure_device() {
    int dev = current_device();
    if (dev < 0) {
        set_last_hip_error("hipGetDevice failed");
        return BSR_ERR_HIP;
    }
    if (dev >= kMaxDevices) return BSR_ERR_UNSUPPORTED;
    DeviceInfo &d = g_devices[dev];
    int st = d.state.load(std::memory_order_acquire);
    if (st == 1) return BSR_OK;
    if (st == -1) return BSR_ERR_ARCH;
    std::lock_guard<std::mutex> lock(g_device_mutex);
    st = d.state.load(std::memory_order_relaxed);
    if (st != 0) return st == 1 ? BSR_OK : BSR_ERR_ARCH;
    hipDeviceProp_t prop;
    hipError_t e = hipGetDeviceProperties(&prop, dev);
    if (e != hipSuccess) {
        set_last_hip_error(hipGetErrorString(e));
        return BSR_ERR_HIP;
    }
    bool ok = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0;
    d.cu_count = prop.multiProcessorCount;
    d.lds_per_block = prop.sharedMemPerBlock;
    d.state.store(ok ? 1 : -1, std::memory_order_release);
    return ok ? BSR_OK : BSR_ERR_ARCH;
}

int auto_slices(int64_t T, const bsr_matrix_t *W, int cu_count) {
    // Enough workgroups to give every CU one: token tiles times slices >= CUs, with at least
    // one block-row per slice.
    const int64_t tiles = (T + 31) / 32;
    const int64_t Nb = W->n_rows / W->R;
    int64_t S = (cu_count > 0 ? cu_count : 256) / (tiles > 0 ? tiles : 1);
    if (S < 1) S = 1;
    if (S > Nb) S = Nb;
    return int(S);
}

int device_cu_count() {
    int dev = current_device();
    return (dev >= 0 && dev < kMaxDevices) ? g_devices[dev].cu_count : 0;
}

size_t device_lds_per_block() {
    int dev = current_device();
    return (dev >= 0 && dev < kMaxDevices) ? g_devices[dev].lds_per_block : 0;
}

}  // namespace bsr

extern "C" {

const char *bsr_last_hip_error(void) { return bsr::g_last_hip_error; }

bsr_status bsr_prune_from_dense(const float *W, int64_t N, int64_t K, int64_t ldw, int32_t R,
                                int32_t C, int64_t k, int32_t *indptr, int32_t *indices,
                                float *data, int64_t capacity_blocks, void *workspace,
                                size_t ws_bytes, void *stream) {
    bsr_status s = bsr::check_prune(W, N, K, ldw, R, C, k, indptr, indices, data,
                                    capacity_blocks, workspace, ws_bytes);
    if (s != BSR_OK) return s;
    if ((s = bsr::ensure_device()) != BSR_OK) return s;
    return bsr::launch_prune(W, N, K, ldw, R, C, k, indptr, indices, data, workspace, stream);
}

bsr_status bsr_spmm_ex(const void *X, bsr_dtype x_dtype, int64_t T, int64_t ldx,
                       const bsr_matrix_t *W, const float *bias, float *Y, int64_t ldy,
                       const bsr_spmm_options_t *opts, void *stream) {
    bsr_status s = bsr::check_spmm(X, int(x_dtype), T, ldx, W, Y, ldy);
    if (s != BSR_OK) return s;
    const int kernel = opts ? opts->kernel : BSR_KERNEL_AUTO;
    const int slices = opts ? opts->slices : 0;
    if (kernel < BSR_KERNEL_AUTO || kernel > BSR_KERNEL_TILED || slices < 0) return BSR_ERR_ARG;
    if (T == 0) return BSR_OK;
    if ((s = bsr::ensure_device()) != BSR_OK) return s;
    if (kernel != BSR_KERNEL_GENERIC && bsr::tiled_supported(W->R, W->C, W->dtype)) {
        const int S = slices > 0 ? slices : bsr::auto_slices(T, W, bsr::device_cu_count());
        bsr::TiledPlan plan =
            bsr::plan_tiled(X, T, ldx, W, S, bsr::device_lds_per_block());
        if (plan.ok) return bsr::launch_spmm_tiled(plan, X, T, ldx, W, bias, Y, ldy, stream);
    }
    if (kernel == BSR_KERNEL_TILED) return BSR_ERR_UNSUPPORTED;
    return bsr::launch_spmm_generic(X, T, ldx, W, bias, Y, ldy, stream);
}

bsr_status bsr_spmm(const void *X, bsr_dtype x_dtype, int64_t T, int64_t ldx,
                    const bsr_matrix_t *W, const float *bias, float *Y, int64_t ldy,
                    void *stream) {
    return bsr_spmm_ex(X, x_dtype, T, ldx, W, bias, Y, ldy, nullptr, stream);
}

bsr_status bsr_to_dense(const bsr_matrix_t *W, float *out, int64_t ldo, void *stream) {
    bsr_status s = bsr::check_to_dense(W, out, ldo);
    if (s != BSR_OK) return s;
    if ((s = bsr::ensure_device()) != BSR_OK) return s;
    return bsr::launch_to_dense(W, out, ldo, stream);
}

bsr_status bsr_cast_f32_bf16(const float *src, uint16_t *dst, int64_t n, void *stream) {
    bsr_status s = bsr::check_cast(src, dst, n);
    if (s != BSR_OK) return s;
    if (n == 0) return BSR_OK;
    if ((s = bsr::ensure_device()) != BSR_OK) return s;
    return bsr::launch_cast(src, dst, n, stream);
}

}  // extern "C"
