// Block-magnitude pruning on the GPU: dense fp32 W -> BSR keeping the top-k blocks.
//
// Sec. 2.1, Eq. 3 partitions W into blocks scored by a per-block norm (l2, or l1: the p = 1 case
// of Eq. 1 and Eq. 2); Eq. 2 bounds the number of nonzero groups, whose projection keeps the k
// blocks of largest norm (globally, or k / Nb in every block-row); Sec. 2.2 stores the result
// as SciPy-style data / indices / indptr.
//
// Three launches on the caller's stream:
//   1. prune_keys_kernel: one thread per block, fp64 key summed sequentially (row r outer,
//      column c inner).  Each fp32 square and each |x| is exact in fp64, so fma(x, x, s) and
//      s + |x| round exactly like the CPU's sequential loop: the key is bit-identical.
//   2. prune_select_kernel: one workgroup.  Radix select over the 64-bit key patterns (keys
//      are >= +0.0, so bit order is value order; NaN is canonicalised above +inf) finds the
//      k-th largest key tau and how many keys equal to tau are kept.  A second sweep in block
//      id order uses workgroup prefix sums to decide each block (key > tau, or key == tau among
//      the first `need_eq` such ids) and to write indptr, indices and the source block ids.
//      Integer LDS atomics count histogram bins, so the result is deterministic.
//      Per-row selection (prune_select_rows_kernel) runs the same radix select and id-order
//      sweep inside each block-row, one workgroup per row; indptr is then i * k_row.
//   3. prune_copy_kernel: one thread per output element copies the kept blocks' bits.
#include <mutex>

#include "device_common.h"

namespace bsr {

namespace {

// The workspace of bsr_prune_from_dense_noalloc: a fixed device array, one copy per GPU.  In
// host code its name is only a stand-in for the symbol; the device address of each GPU's copy
// comes from hipGetSymbolAddress, looked up once per device with that device current.
__device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

constexpr int kScratchDevices = 64;
void *g_scratch_ptr[kScratchDevices] = {};
std::mutex g_scratch_mutex;

constexpr int kKeyThreads = 256;
constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / 64;
constexpr unsigned long long kNaNKey = 0x7FF8000000000000ull;

template <bool kL1>
__global__ __launch_bounds__(kKeyThreads) void prune_keys_kernel(
    const float *__restrict__ W, int64_t ldw, int32_t R, int32_t C, int64_t Kb, int64_t nb,
    unsigned long long *__restrict__ keybits) {
    const int64_t b = int64_t(blockIdx.x) * kKeyThreads + threadIdx.x;
    if (b >= nb) return;
    const int64_t i = b / Kb, j = b - i * Kb;
    const float *base = W + (i * R) * ldw + j * C;
    double s = 0.0;
    for (int r = 0; r < R; ++r) {
        const float *row = base + int64_t(r) * ldw;
        for (int c = 0; c < C; ++c) {
            const double x = static_cast<double>(row[c]);
            if constexpr (kL1) s = __dadd_rn(s, fabs(x));
            else s = __fma_rn(x, x, s);
        }
    }
    unsigned long long u = static_cast<unsigned long long>(__double_as_longlong(s));
    if (s != s) u = kNaNKey;
    keybits[b] = u;
}

// Exclusive prefix count of `pred` over the workgroup of NWAVES waves (thread order) and its
// total.
template <int NWAVES = kSelWaves>
__device__ __forceinline__ void wg_scan(bool pred, unsigned &excl, unsigned &total,
                                        unsigned *wave_tot) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const unsigned long long m = __ballot(pred);
    const unsigned long long below = lane ? (m & ((1ull << lane) - 1ull)) : 0ull;
    const unsigned in_wave = static_cast<unsigned>(__popcll(below));
    if (lane == 0) wave_tot[wave] = static_cast<unsigned>(__popcll(m));
    __syncthreads();
    unsigned before = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < NWAVES; ++w) {
        const unsigned c = wave_tot[w];
        before += (w < wave) ? c : 0u;
        tot += c;
    }
    __syncthreads();
    excl = before + in_wave;
    total = tot;
}

__global__ __launch_bounds__(kSelThreads) void prune_select_kernel(
    const unsigned long long *__restrict__ keybits, int64_t nb, int64_t Kb, int64_t Nb,
    int64_t k, int32_t *__restrict__ indptr, int32_t *__restrict__ indices,
    int32_t *__restrict__ src) {
    __shared__ unsigned hist[256];
    __shared__ unsigned wave_tot[kSelWaves];
    __shared__ unsigned long long s_prefix;
    __shared__ long long s_remaining;
    const int tid = threadIdx.x;

    if (k <= 0) {
        for (int64_t i = tid; i <= Nb; i += kSelThreads) indptr[i] = 0;
        return;
    }

    // Radix select of the k-th largest key, 8 bits per pass from the top.
    unsigned long long prefix = 0, pmask = 0;
    long long remaining = k;  // rank of the target among keys matching `prefix` (1-based)
    for (int pass = 0; pass < 8; ++pass) {
        const int shift = 56 - 8 * pass;
        if (tid < 256) hist[tid] = 0;
        __syncthreads();
        for (int64_t b = tid; b < nb; b += kSelThreads) {
            const unsigned long long u = keybits[b];
            if ((u & pmask) == prefix) atomicAdd(&hist[(u >> shift) & 255ull], 1u);
        }
        __syncthreads();
        if (tid == 0) {
            long long cum = 0;
            int digit = 0;
            for (int v = 255; v >= 0; --v) {
                const long long h = hist[v];
                if (cum + h >= remaining) {
                    digit = v;
                    break;
                }
                cum += h;
            }
            s_prefix = prefix | (static_cast<unsigned long long>(digit) << shift);
            s_remaining = remaining - cum;
        }
        __syncthreads();
        prefix = s_prefix;
        remaining = s_remaining;
        pmask |= 0xFFull << shift;
        __syncthreads();
    }
    const unsigned long long tau = prefix;
    const long long need_eq = remaining;  // keys == tau to keep, lowest ids first

    // Decide and place every block in id order (ids are row-major, so the kept blocks come out
    // sorted by block-row and then by block-column, as the BSR layout requires).
    long long run_eq = 0, run_keep = 0;
    for (int64_t base = 0; base < nb; base += kSelThreads) {
        const int64_t b = base + tid;
        const bool valid = b < nb;
        const unsigned long long u = valid ? keybits[b] : 0ull;
        const bool gt = valid && u > tau;
        const bool eq = valid && u == tau;
        unsigned eq_ex, eq_tot;
        wg_scan(eq, eq_ex, eq_tot, wave_tot);
        const bool keep = gt || (eq && (run_eq + static_cast<long long>(eq_ex)) < need_eq);
        unsigned keep_ex, keep_tot;
        wg_scan(keep, keep_ex, keep_tot, wave_tot);
        const long long pos = run_keep + static_cast<long long>(keep_ex);
        if (valid) {
            const int64_t i = b / Kb, j = b - i * Kb;
            if (keep) {
                indices[pos] = static_cast<int32_t>(j);
                src[pos] = static_cast<int32_t>(b);
            }
            if (j == 0) indptr[i] = static_cast<int32_t>(pos);
        }
        run_eq += eq_tot;
        run_keep += keep_tot;
    }
    if (tid == 0) indptr[Nb] = static_cast<int32_t>(k);
}

constexpr int kRowThreads = 256;
constexpr int kRowWaves = kRowThreads / 64;

// Per-row selection: workgroup i keeps the k_row blocks of block-row i that come first in the
// order (key descending, column ascending), with the radix select and id-order sweep of
// prune_select_kernel restricted to the row.  Every row keeps k_row blocks, so indptr[i] is
// i * k_row and the kept blocks of row i occupy positions i * k_row .. (i + 1) * k_row - 1.
__global__ __launch_bounds__(kRowThreads) void prune_select_rows_kernel(
    const unsigned long long *__restrict__ keybits, int64_t Kb, int64_t Nb, int64_t k_row,
    int32_t *__restrict__ indptr, int32_t *__restrict__ indices, int32_t *__restrict__ src) {
    __shared__ unsigned hist[256];
    __shared__ unsigned wave_tot[kRowWaves];
    __shared__ unsigned long long s_prefix;
    __shared__ long long s_remaining;
    const int tid = threadIdx.x;
    const int64_t i = blockIdx.x;
    if (tid == 0) {
        indptr[i] = static_cast<int32_t>(i * k_row);
        if (i == Nb - 1) indptr[Nb] = static_cast<int32_t>(Nb * k_row);
    }
    if (k_row <= 0) return;   // uniform: a kernel argument
    const unsigned long long *key = keybits + i * Kb;

    unsigned long long prefix = 0, pmask = 0;
    long long remaining = k_row;
    for (int pass = 0; pass < 8; ++pass) {
        const int shift = 56 - 8 * pass;
        hist[tid] = 0;   // kRowThreads == 256 bins
        __syncthreads();
        for (int64_t b = tid; b < Kb; b += kRowThreads) {
            const unsigned long long u = key[b];
            if ((u & pmask) == prefix) atomicAdd(&hist[(u >> shift) & 255ull], 1u);
        }
        __syncthreads();
        if (tid == 0) {
            long long cum = 0;
            int digit = 0;
            for (int v = 255; v >= 0; --v) {
                const long long h = hist[v];
                if (cum + h >= remaining) {
                    digit = v;
                    break;
                }
                cum += h;
            }
            s_prefix = prefix | (static_cast<unsigned long long>(digit) << shift);
            s_remaining = remaining - cum;
        }
        __syncthreads();
        prefix = s_prefix;
        remaining = s_remaining;
        pmask |= 0xFFull << shift;
        __syncthreads();
    }
    const unsigned long long tau = prefix;
    const long long need_eq = remaining;

    long long run_eq = 0, run_keep = 0;
    for (int64_t base = 0; base < Kb; base += kRowThreads) {
        const int64_t j = base + tid;
        const bool valid = j < Kb;
        const unsigned long long u = valid ? key[j] : 0ull;
        const bool gt = valid && u > tau;
        const bool eq = valid && u == tau;
        unsigned eq_ex, eq_tot;
        wg_scan<kRowWaves>(eq, eq_ex, eq_tot, wave_tot);
        const bool keep = gt || (eq && (run_eq + static_cast<long long>(eq_ex)) < need_eq);
        unsigned keep_ex, keep_tot;
        wg_scan<kRowWaves>(keep, keep_ex, keep_tot, wave_tot);
        const long long pos = i * k_row + run_keep + static_cast<long long>(keep_ex);
        if (keep) {
            indices[pos] = static_cast<int32_t>(j);
            src[pos] = static_cast<int32_t>(i * Kb + j);
        }
        run_eq += eq_tot;
        run_keep += keep_tot;
    }
}

__global__ __launch_bounds__(256) void prune_copy_kernel(
    const float *__restrict__ W, int64_t ldw, int32_t R, int32_t C, int64_t Kb, int64_t nb,
    int64_t k, const int32_t *__restrict__ src, float *__restrict__ data) {
    const int64_t RC = int64_t(R) * C;
    const int64_t total = k * RC;
    const unsigned *Wu = reinterpret_cast<const unsigned *>(W);
    unsigned *Du = reinterpret_cast<unsigned *>(data);
    for (int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x; e < total;
         e += int64_t(gridDim.x) * 256) {
        const int64_t p = e / RC, rc = e - p * RC;
        const int64_t r = rc / C, c = rc - r * C;
        const int64_t b = clamp64(src[p], 0, nb - 1);
        const int64_t i = b / Kb, j = b - i * Kb;
        Du[e] = Wu[(i * R + r) * ldw + j * C + c];
    }
}

}  // namespace

bsr_status noalloc_scratch(void **ptr) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) {
        set_last_hip_error(hipGetErrorString(e));
        return BSR_ERR_HIP;
    }
    if (dev < 0 || dev >= kScratchDevices) return BSR_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (g_scratch_ptr[dev] == nullptr) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || p == nullptr) {
            set_last_hip_error(e != hipSuccess ? hipGetErrorString(e)
                                               : "hipGetSymbolAddress returned NULL");
            return BSR_ERR_HIP;
        }
        g_scratch_ptr[dev] = p;
    }
    *ptr = g_scratch_ptr[dev];
    return BSR_OK;
}

bsr_status launch_prune(const float *W, int64_t N, int64_t K, int64_t ldw, int32_t R, int32_t C,
                        int64_t k, int32_t *indptr, int32_t *indices, float *data,
                        void *workspace, int norm, int select, void *stream) {
    const int64_t Nb = N / R, Kb = K / C, nb = Nb * Kb;
    const PruneWorkspace ws = prune_workspace_layout(nb);
    char *base = static_cast<char *>(workspace);
    auto *keybits = reinterpret_cast<unsigned long long *>(base + ws.key_offset);
    auto *src = reinterpret_cast<int32_t *>(base + ws.src_offset);
    hipStream_t st = as_stream(stream);

    if (k > 0) {
        const unsigned g = static_cast<unsigned>((nb + kKeyThreads - 1) / kKeyThreads);
        auto keys = norm == BSR_NORM_L1 ? prune_keys_kernel<true> : prune_keys_kernel<false>;
        hipLaunchKernelGGL(keys, dim3(g), dim3(kKeyThreads), 0, st, W, ldw, R, C, Kb, nb,
                           keybits);
        bsr_status s = launch_status();
        if (s != BSR_OK) return s;
    }
    if (select == BSR_SELECT_PER_ROW)
        hipLaunchKernelGGL(prune_select_rows_kernel, dim3(static_cast<unsigned>(Nb)),
                           dim3(kRowThreads), 0, st, keybits, Kb, Nb, k / Nb, indptr, indices,
                           src);
    else
        hipLaunchKernelGGL(prune_select_kernel, dim3(1), dim3(kSelThreads), 0, st, keybits, nb,
                           Kb, Nb, k, indptr, indices, src);
    bsr_status s = launch_status();
    if (s != BSR_OK || k == 0) return s;
    hipLaunchKernelGGL(prune_copy_kernel, dim3(grid_for(k * R * C, 256)), dim3(256), 0, st, W,
                       ldw, R, C, Kb, nb, k, src, data);
    return launch_status();
}

}  // namespace bsr
