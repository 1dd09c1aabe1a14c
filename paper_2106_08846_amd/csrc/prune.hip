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
//   2. prune_select_kernel (prune_select_reg_kernel when the keys fit in the workgroup's
//      registers): one workgroup.  Radix select over the 64-bit key patterns (keys
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

// One radix step of the selection, by the first wave, lane l holding the counts c of bins
// 4 l .. 4 l + 3 (the bins of this digit of the keys that match the prefix so far): the digit
// of the key with rank `remaining` (1-based, descending), i.e. the largest v whose bins
// v .. 255 hold at least `remaining` keys.  Suffix sums over the lanes give each bin's count
// of keys at or above it.  Writes the extended prefix and the rank within bin v.
__device__ __forceinline__ void pick_digit_counts(const unsigned (&c)[4], long long remaining,
                                                  unsigned long long prefix, int shift,
                                                  unsigned long long *s_prefix,
                                                  long long *s_remaining) {
    const int lane = threadIdx.x & 63;
    const unsigned t = c[0] + c[1] + c[2] + c[3];
    unsigned sfx = t;   // keys in the bins of lanes >= lane
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const unsigned y = __shfl_down(sfx, d);
        sfx += lane + d < 64 ? y : 0u;
    }
    long long at[4];    // keys in bins >= 4 lane + q
    at[3] = static_cast<long long>(sfx - t) + c[3];
    at[2] = at[3] + c[2];
    at[1] = at[2] + c[1];
    at[0] = at[1] + c[0];
    const int qb = at[3] >= remaining ? 3 : at[2] >= remaining ? 2
                 : at[1] >= remaining ? 1 : at[0] >= remaining ? 0 : -1;
    const unsigned long long m = __ballot(qb >= 0);
    if (m == 0ull) {   // fewer keys than the rank (not reached for 1 <= k <= nb)
        if (lane == 0) {
            *s_prefix = prefix;
            *s_remaining = remaining - static_cast<long long>(sfx);
        }
        return;
    }
    const int L = 63 - __clzll(static_cast<long long>(m));
    if (lane == L) {
        const int digit = 4 * lane + qb;
        *s_prefix = prefix | (static_cast<unsigned long long>(digit) << shift);
        *s_remaining = remaining - (at[qb] - static_cast<long long>(c[qb]));
    }
}

__device__ __forceinline__ void pick_digit(const unsigned *hist, long long remaining,
                                           unsigned long long prefix, int shift,
                                           unsigned long long *s_prefix,
                                           long long *s_remaining) {
    const int lane = threadIdx.x & 63;
    unsigned c[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) c[q] = hist[4 * lane + q];
    pick_digit_counts(c, remaining, prefix, shift, s_prefix, s_remaining);
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
        if (tid < 64) pick_digit(hist, remaining, prefix, shift, &s_prefix, &s_remaining);
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

// prune_select_kernel for nb <= kSelThreads * kRegKeys (e.g. a 1024 x 1024 weight in 32 x 1
// blocks): the same selection (radix select of tau, then the keys > tau and the first need_eq
// keys == tau in id order) with every key read once, coalesced, into registers: thread t holds
// ids t + kSelThreads e, e < kRegKeys ("round" e).
//   * The high bytes that every key shares (min and max agree on them) are not radix passes.
//   * Histogram bins are spread over kHistCopies copies (lane mod kHistCopies), kHistPitch =
//     257 words apart, because the keys of one matrix crowd into few bins: one bin's copies then
//     sit in different LDS banks.  The first wave sums the copies (and clears them for the next
//     pass) and picks the digit, so a pass costs two barriers.
//   * Placement: per round and wave, the counts of equal keys and then of kept keys go to a
//     table of kRegKeys x kSelWaves entries whose exclusive prefix, in (round, wave) order, is id
//     order; a key's rank is its table entry plus the lanes below it in its wave.
constexpr int kRegKeys = 32;
constexpr int kHistCopies = 16;
constexpr int kHistPitch = 257;
constexpr int kTab = kRegKeys * kSelWaves;   // 512

// Exclusive prefix, in place, of tab[kTab] by the first wave (8 entries per lane).
__device__ __forceinline__ void tab_excl_scan(unsigned *tab) {
    const int lane = threadIdx.x & 63;
    unsigned v[8], t = 0;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        v[q] = tab[8 * lane + q];
        t += v[q];
    }
    unsigned incl = t;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const unsigned y = __shfl_up(incl, d);
        incl += lane >= d ? y : 0u;
    }
    unsigned run = incl - t;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        tab[8 * lane + q] = run;
        run += v[q];
    }
}

__global__ __launch_bounds__(kSelThreads) void prune_select_reg_kernel(
    const unsigned long long *__restrict__ keybits, int64_t nb, int64_t Kb, int64_t Nb,
    int64_t k, int32_t *__restrict__ indptr, int32_t *__restrict__ indices,
    int32_t *__restrict__ src) {
    __shared__ unsigned hist[kHistCopies * kHistPitch];
    __shared__ unsigned tab[kTab];
    __shared__ unsigned long long s_min[kSelWaves], s_max[kSelWaves];
    __shared__ unsigned long long s_prefix;
    __shared__ long long s_remaining;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

    if (k <= 0) {
        for (int64_t i = tid; i <= Nb; i += kSelThreads) indptr[i] = 0;
        return;
    }
    const int n = int(nb);
    // All loads are issued before any is used: range-checked buffer loads (ids past nb read
    // 0 and touch no memory) need no branch per key.
    unsigned long long key[kRegKeys];
    {
        const __amdgpu_buffer_rsrc_t rk = buffer_rsrc(keybits, unsigned(n) * 8u);
#pragma unroll
        for (int e = 0; e < kRegKeys; ++e) {
            const auto w = __builtin_amdgcn_raw_buffer_load_b64(rk, (tid + kSelThreads * e) * 8,
                                                                0, 0);
            key[e] = (static_cast<unsigned long long>(w[1]) << 32) | w[0];
        }
    }
    for (int i = tid; i < kHistCopies * kHistPitch; i += kSelThreads) hist[i] = 0;
    unsigned long long kmin = ~0ull, kmax = 0ull;
#pragma unroll
    for (int e = 0; e < kRegKeys; ++e) {
        if (tid + kSelThreads * e < n) {
            kmin = key[e] < kmin ? key[e] : kmin;
            kmax = key[e] > kmax ? key[e] : kmax;
        }
    }
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) {
        const unsigned long long x = __shfl_xor(kmin, d), y = __shfl_xor(kmax, d);
        kmin = x < kmin ? x : kmin;
        kmax = y > kmax ? y : kmax;
    }
    if (lane == 0) {
        s_min[wave] = kmin;
        s_max[wave] = kmax;
    }
    __syncthreads();
    kmin = ~0ull;
    kmax = 0ull;
#pragma unroll
    for (int w = 0; w < kSelWaves; ++w) {
        kmin = s_min[w] < kmin ? s_min[w] : kmin;
        kmax = s_max[w] > kmax ? s_max[w] : kmax;
    }
    // Leading bytes shared by every key: all keys match them, so the select's prefix there is
    // that of any key and the rank is unchanged.
    int pass0 = 0;
    while (pass0 < 8 && ((kmin ^ kmax) >> (56 - 8 * pass0)) == 0) ++pass0;
    const unsigned long long shared_mask = pass0 == 0 ? 0ull : ~0ull << (64 - 8 * pass0);
    unsigned long long prefix = kmin & shared_mask, pmask = shared_mask;
    long long remaining = k;
    unsigned *h = hist + (lane % kHistCopies) * kHistPitch;
    for (int pass = pass0; pass < 8; ++pass) {
        const int shift = 56 - 8 * pass;
#pragma unroll
        for (int e = 0; e < kRegKeys; ++e)
            if (tid + kSelThreads * e < n && (key[e] & pmask) == prefix)
                atomicAdd(&h[(key[e] >> shift) & 255ull], 1u);
        __syncthreads();
        if (wave == 0) {
            unsigned c[4] = {0u, 0u, 0u, 0u};
#pragma unroll
            for (int cp = 0; cp < kHistCopies; ++cp) {
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    c[q] += hist[cp * kHistPitch + 4 * lane + q];
                    hist[cp * kHistPitch + 4 * lane + q] = 0;
                }
            }
            pick_digit_counts(c, remaining, prefix, shift, &s_prefix, &s_remaining);
        }
        __syncthreads();
        prefix = s_prefix;
        remaining = s_remaining;
        pmask |= 0xFFull << shift;
    }
    const unsigned long long tau = prefix;
    const long long need_eq = remaining;   // keys == tau to keep, lowest ids first

    const unsigned long long below = (1ull << lane) - 1ull;   // lanes under this one
    unsigned eqm = 0, gtm = 0;
#pragma unroll
    for (int e = 0; e < kRegKeys; ++e) {
        const bool v = tid + kSelThreads * e < n;
        eqm |= (v && key[e] == tau) ? 1u << e : 0u;
        gtm |= (v && key[e] > tau) ? 1u << e : 0u;
    }
    // Ranks of the equal keys in id order.
#pragma unroll
    for (int e = 0; e < kRegKeys; ++e) {
        const unsigned long long b = __ballot((eqm >> e) & 1u);
        if (lane == 0) tab[e * kSelWaves + wave] = unsigned(__popcll(b));
    }
    __syncthreads();
    if (wave == 0) tab_excl_scan(tab);
    __syncthreads();
    unsigned keepm = gtm;
#pragma unroll
    for (int e = 0; e < kRegKeys; ++e) {
        const unsigned long long b = __ballot((eqm >> e) & 1u);
        const long long rank = static_cast<long long>(tab[e * kSelWaves + wave]) +
                               __popcll(b & below);
        keepm |= ((eqm >> e) & 1u) && rank < need_eq ? 1u << e : 0u;
    }
    __syncthreads();   // every wave has read the equal-key ranks
    // Positions of the kept keys in id order.
#pragma unroll
    for (int e = 0; e < kRegKeys; ++e) {
        const unsigned long long b = __ballot((keepm >> e) & 1u);
        if (lane == 0) tab[e * kSelWaves + wave] = unsigned(__popcll(b));
    }
    __syncthreads();
    if (wave == 0) tab_excl_scan(tab);
    __syncthreads();
    const unsigned kb = unsigned(Kb);
#pragma unroll
    for (int e = 0; e < kRegKeys; ++e) {
        const unsigned id = unsigned(tid + kSelThreads * e);
        const unsigned long long b = __ballot((keepm >> e) & 1u);
        if (id < unsigned(n)) {
            const int pos = int(tab[e * kSelWaves + wave]) + __popcll(b & below);
            const unsigned i = id / kb, j = id - i * kb;
            if (j == 0) indptr[i] = pos;
            if ((keepm >> e) & 1u) {
                indices[pos] = int32_t(j);
                src[pos] = int32_t(id);
            }
        }
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
        if (tid < 64) pick_digit(hist, remaining, prefix, shift, &s_prefix, &s_remaining);
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
    else if (nb <= int64_t(kSelThreads) * kRegKeys)
        hipLaunchKernelGGL(prune_select_reg_kernel, dim3(1), dim3(kSelThreads), 0, st, keybits,
                           nb, Kb, Nb, k, indptr, indices, src);
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
