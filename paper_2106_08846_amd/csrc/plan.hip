// Per-matrix product plans (the paper's compiler keeps a buffer of sparse operators and reuses
// tasks with identical sparse structure, Sec. 2.2, third bullet): the part of a BSR product
// that depends only on the matrix, prepared once on the device.
//
// For linear 32x1 blocks a plan holds, in one caller-owned buffer:
//   * uptr int32[Nb + 1]: the first unit of every block-row, where a row of n stored blocks
//     has ceil(n / KB) units of KB consecutive blocks (KB = 8 for fp32 on fp32 matrix cores,
//     16 for bf16 and for fp32 split into bf16 pieces);
//   * the columns of every unit, in the order the flat kernel's lanes read them, as byte
//     offsets into the X tile, with the tile's zero pad column (index Kb) for the blocks a row's
//     last unit lacks;
//   * the weights of every unit, in the lane order of its MFMA B operands (zero for missing
//     blocks); with split arithmetic, the three bf16 pieces of every weight, one operand plane
//     per piece.
// Two launches: one workgroup scans the per-row unit counts into uptr, then one thread per
// (unit, lane) finds its row by binary search over uptr and packs its columns and weights.
// The layout reserves ceil(nnzb / KB) + Nb units (a row wastes less than one unit); units past
// the last are filled with pad columns and zero weights.
#include "device_common.h"
#include "spmm_tiled.h"
#include "spmm_units.h"

namespace bsr {

namespace {

constexpr int kScanThreads = 1024;

// uptr[i + 1] = uptr[i] + ceil((indptr[i + 1] - indptr[i]) / KB), uptr[0] = 0; indptr entries
// are clamped to [0, nnzb] (and a decreasing pair counts as an empty row), as the product
// kernels read them.
__global__ __launch_bounds__(kScanThreads) void plan_uptr_kernel(
    const int32_t *__restrict__ indptr, int Nb, int nnzb, int KB, int32_t *__restrict__ uptr) {
    __shared__ int s_wave[kScanThreads / 64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int carry = 0;
    if (threadIdx.x == 0) uptr[0] = 0;
    for (int base = 0; base < Nb; base += kScanThreads) {
        const int i = base + threadIdx.x;
        int cnt = 0;
        if (i < Nb) {
            const int n = clampi(indptr[i + 1], 0, nnzb) - clampi(indptr[i], 0, nnzb);
            cnt = n > 0 ? (n + KB - 1) / KB : 0;
        }
        int incl = cnt;   // inclusive scan within the wave
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int y = __shfl_up(incl, d, 64);
            if (lane >= d) incl += y;
        }
        if (lane == 63) s_wave[wave] = incl;
        __syncthreads();
        int before = carry;
        for (int w = 0; w < wave; ++w) before += s_wave[w];
        if (i < Nb) uptr[i + 1] = before + incl;
        int total = 0;
        for (int w = 0; w < kScanThreads / 64; ++w) total += s_wave[w];
        carry += total;
        __syncthreads();
    }
}

// Row of unit u: the last row i < Nb with uptr[i] <= u (rows before it end at or before u).
__device__ __forceinline__ int unit_row(const int32_t *__restrict__ uptr, int Nb, int u) {
    int lo = 0, hi = Nb - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (uptr[mid] <= u) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

// One thread per (unit, lane).  Native fp32 (KIND 0): lane l packs weights of blocks 2m + l/32
// (m = 0..3), feature l%32, and lanes 0..7 pack the columns cols[u][h][m] (block 2m + h).
// Native bf16 (KIND 1): lane l packs blocks 8(l/32) + e (e = 0..7), feature l%32, and lanes
// 0..15 pack the columns cols[u][h][c][s] (block 8h + 4s + c).  Split fp32 (KIND 2): lane l
// packs the three bf16 pieces of blocks 8(l/32) + e, feature l%32, one plane per piece, and
// lanes 0..15 pack the uint16 columns cols[u][h][e] (block 8h + e).
template <int KIND>
__global__ __launch_bounds__(256) void plan_fill_kernel(
    const int32_t *__restrict__ indptr, const int32_t *__restrict__ indices,
    const void *__restrict__ data, int Nb, int nnzb, int Kb, const int32_t *__restrict__ uptr,
    int64_t max_units, int32_t *__restrict__ ucol, void *__restrict__ uval) {
    constexpr bool BF = KIND == 1;
    constexpr int KB = KIND == 0 ? 8 : 16;
    const int64_t total = max_units * 64;
    for (int64_t t = int64_t(blockIdx.x) * 256 + threadIdx.x; t < total;
         t += int64_t(gridDim.x) * 256) {
        const int u = int(t >> 6), l = int(t & 63), h = l >> 5, f = l & 31;
        const int units = clampi(uptr[Nb], 0, int(max_units));
        int p0 = 0, e = 0;   // blocks [p0, e) of the unit (empty past the last unit)
        if (u < units) {
            const int r = unit_row(uptr, Nb, u);
            const int b0 = clampi(indptr[r], 0, nnzb), b1 = clampi(indptr[r + 1], 0, nnzb);
            p0 = b0 + KB * (u - uptr[r]);
            e = b1;
        }
        // A block's column as the byte offset the kernel's gather adds: scale * column, the
        // column clamped to [0, Kb] (Kb, the tile's zero pad column, for missing blocks).
        constexpr int kScale = KIND == 0   ? PlanUnit<32, 1, false>::kColScale
                               : KIND == 1 ? PlanUnit<32, 1, true>::kColScale
                                           : SplitPlanUnit::kColScale;
        auto col = [&](int p) -> int32_t {
            return kScale * (p < e ? int32_t(min(unsigned(indices[p]), unsigned(Kb))) : int32_t(Kb));
        };
        if constexpr (KIND == 2) {
            const float *d = static_cast<const float *>(data);
            uint16_t w[3][8];
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const int p = p0 + 8 * h + q;
                const unsigned v = p < e ? __float_as_uint(d[int64_t(p) * 32 + f]) : 0u;
                const float rr = __uint_as_float(v) - __uint_as_float(v & 0xffff0000u);
                const float cc = rr - __uint_as_float(__float_as_uint(rr) & 0xffff0000u);
                w[0][q] = uint16_t(v >> 16);
                w[1][q] = uint16_t(__float_as_uint(rr) >> 16);
                w[2][q] = uint16_t(__float_as_uint(cc) >> 16);
            }
            uint16_t *dst = reinterpret_cast<uint16_t *>(static_cast<char *>(uval) +
                                                         int64_t(u) * SplitPlanUnit::kValBytes) +
                            l * 8;
#pragma unroll
            for (int pc = 0; pc < 3; ++pc)
#pragma unroll
                for (int q = 0; q < 8; ++q) dst[pc * (SplitPlanUnit::kPlaneBytes / 2) + q] = w[pc][q];
            if (l < 16) {   // cols[u][hh][q] = block 8 hh + q
                const int hh = l >> 3, q = l & 7;
                reinterpret_cast<uint16_t *>(ucol)[int64_t(u) * 16 + l] =
                    uint16_t(col(p0 + 8 * hh + q));
            }
        } else if constexpr (BF) {
            const uint16_t *d = static_cast<const uint16_t *>(data);
            uint16_t w[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const int p = p0 + 8 * h + q;
                w[q] = p < e ? d[int64_t(p) * 32 + f] : uint16_t(0);
            }
            uint16_t *dst = static_cast<uint16_t *>(uval) + (int64_t(u) * 64 + l) * 8;
#pragma unroll
            for (int q = 0; q < 8; ++q) dst[q] = w[q];
            if (l < 16) {   // cols[u][hh][c][s] = block 8 hh + 4 s + c
                const int hh = l >> 3, c = (l >> 1) & 3, sidx = l & 1;
                ucol[int64_t(u) * 16 + l] = col(p0 + 8 * hh + 4 * sidx + c);
            }
        } else {
            const float *d = static_cast<const float *>(data);
            float w[4];
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                const int p = p0 + 2 * m + h;
                w[m] = p < e ? d[int64_t(p) * 32 + f] : 0.0f;
            }
            float *dst = static_cast<float *>(uval) + (int64_t(u) * 64 + l) * 4;
#pragma unroll
            for (int m = 0; m < 4; ++m) dst[m] = w[m];
            if (l < 8) {   // cols[u][hh][m] = block 2 m + hh
                const int hh = l >> 2, m = l & 3;
                ucol[int64_t(u) * 8 + l] = col(p0 + 2 * m + hh);
            }
        }
    }
}

int64_t align256(int64_t x) { return (x + 255) & ~int64_t(255); }

}  // namespace

PlanLayout plan_layout(const bsr_matrix_t *W, int arith) {
    PlanLayout L{};
    if (!plan_supported(W->R, W->C, W->dtype, arith)) return L;
    const bool bf = W->dtype == BSR_BF16;
    L.arith = resolve_arith(W->dtype, arith);
    const bool split = L.arith == BSR_ARITH_BF16X3;
    // Split plans store columns as 16-bit byte offsets into a row of the fp32 X tile.
    if (split && (W->n_cols / W->C) * SplitPlanUnit::kColScale > SplitPlanUnit::kMaxColBytes)
        return L;
    L.unit_blocks = split ? SplitPlanUnit::KB : bf ? PlanUnit<32, 1, true>::KB : PlanUnit<32, 1, false>::KB;
    const int64_t Nb = W->n_rows / W->R;
    L.max_units = (W->nnzb + L.unit_blocks - 1) / L.unit_blocks + Nb;
    const int64_t col_bytes = split ? SplitPlanUnit::kColBytes
                              : bf  ? PlanUnit<32, 1, true>::kColBytes
                                    : PlanUnit<32, 1, false>::kColBytes;
    const int64_t val_bytes = split ? SplitPlanUnit::kValBytes
                              : bf  ? PlanUnit<32, 1, true>::kValBytes
                                    : PlanUnit<32, 1, false>::kValBytes;
    L.uptr_offset = 0;
    L.col_offset = align256((Nb + 1) * 4);
    L.val_offset = L.col_offset + align256(L.max_units * col_bytes);
    L.total = L.val_offset + align256(L.max_units * val_bytes);
    return L;
}

bsr_status launch_plan_prepare(const bsr_matrix_t *W, void *mem, const PlanLayout &L,
                               void *stream) {
    hipStream_t st = as_stream(stream);
    char *base = static_cast<char *>(mem);
    int32_t *uptr = reinterpret_cast<int32_t *>(base + L.uptr_offset);
    int32_t *ucol = reinterpret_cast<int32_t *>(base + L.col_offset);
    void *uval = base + L.val_offset;
    const int Nb = int(W->n_rows / W->R), nnzb = int(W->nnzb), Kb = int(W->n_cols / W->C);
    hipLaunchKernelGGL(plan_uptr_kernel, dim3(1), dim3(kScanThreads), 0, st, W->indptr, Nb,
                       nnzb, L.unit_blocks, uptr);
    bsr_status s = launch_status();
    if (s != BSR_OK) return s;
    const unsigned g = grid_for(L.max_units * 64, 256);
    if (L.arith == BSR_ARITH_BF16X3)
        hipLaunchKernelGGL(plan_fill_kernel<2>, dim3(g), dim3(256), 0, st, W->indptr,
                           W->indices, W->data, Nb, nnzb, Kb, uptr, L.max_units, ucol, uval);
    else if (W->dtype == BSR_BF16)
        hipLaunchKernelGGL(plan_fill_kernel<1>, dim3(g), dim3(256), 0, st, W->indptr,
                           W->indices, W->data, Nb, nnzb, Kb, uptr, L.max_units, ucol, uval);
    else
        hipLaunchKernelGGL(plan_fill_kernel<0>, dim3(g), dim3(256), 0, st, W->indptr,
                           W->indices, W->data, Nb, nnzb, Kb, uptr, L.max_units, ucol, uval);
    return launch_status();
}

}  // namespace bsr
