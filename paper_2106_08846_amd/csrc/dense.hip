// BSR -> dense expansion and the fp32 -> bf16 cast.
#include "device_common.h"

namespace bsr {

namespace {

// out[n][k] = stored element covering (n, k), else +0.0.  One thread per dense element; the
// block is found by binary search over the (ascending) indices of its block-row.  Bits are
// copied unchanged.
__global__ __launch_bounds__(256) void to_dense_kernel(
    const int32_t *__restrict__ indptr, const int32_t *__restrict__ indices,
    const unsigned *__restrict__ data, int64_t nnzb, int64_t N, int64_t K, int32_t R, int32_t C,
    int64_t Kb, unsigned *__restrict__ out, int64_t ldo) {
    const int64_t total = N * K;
    for (int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x; e < total;
         e += int64_t(gridDim.x) * 256) {
        const int64_t n = e / K, kk = e - n * K;
        const int64_t i = n / R, r = n - i * R;
        const int64_t j = kk / C, c = kk - j * C;
        int64_t lo = clamp64(indptr[i], 0, nnzb);
        int64_t hi = clamp64(indptr[i + 1], lo, nnzb);
        unsigned v = 0u;
        while (lo < hi) {
            const int64_t mid = (lo + hi) >> 1;
            const int32_t jm = indices[mid];
            if (jm < j) {
                lo = mid + 1;
            } else if (jm > j) {
                hi = mid;
            } else {
                v = data[(mid * R + r) * C + c];
                break;
            }
        }
        out[n * ldo + kk] = v;
    }
}

// Round to nearest, ties to even, on the bit pattern: adding 0x7FFF plus the lowest kept bit
// carries into the kept half exactly when the dropped half is above one half ulp, or equal to it
// with an odd kept half.  NaN keeps its upper half with the quiet bit set.
__global__ __launch_bounds__(256) void cast_f32_bf16_kernel(const unsigned *__restrict__ src,
                                                            unsigned short *__restrict__ dst,
                                                            int64_t n) {
    for (int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x; e < n;
         e += int64_t(gridDim.x) * 256) {
        const unsigned u = src[e];
        unsigned h;
        if ((u & 0x7FFFFFFFu) > 0x7F800000u) {
            h = (u >> 16) | 0x0040u;
        } else {
            h = (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
        }
        dst[e] = static_cast<unsigned short>(h);
    }
}

}  // namespace

bsr_status launch_to_dense(const bsr_matrix_t *W, float *out, int64_t ldo, void *stream) {
    const int64_t N = W->n_rows, K = W->n_cols, Kb = K / W->C;
    hipLaunchKernelGGL(to_dense_kernel, dim3(grid_for(N * K, 256)), dim3(256), 0,
                       as_stream(stream), W->indptr, W->indices,
                       static_cast<const unsigned *>(W->data), W->nnzb, N, K, W->R, W->C, Kb,
                       reinterpret_cast<unsigned *>(out), ldo);
    return launch_status();
}

bsr_status launch_cast(const float *src, uint16_t *dst, int64_t n, void *stream) {
    hipLaunchKernelGGL(cast_f32_bf16_kernel, dim3(grid_for(n, 256)), dim3(256), 0,
                       as_stream(stream), reinterpret_cast<const unsigned *>(src),
                       reinterpret_cast<unsigned short *>(dst), n);
    return launch_status();
}

}  // namespace bsr
