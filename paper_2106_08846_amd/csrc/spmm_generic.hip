// Reference-shaped BSR product: one thread per output element, any block shape, fp32 or bf16.
//
// Y[t][n] = bias[n] + sum over the stored blocks p of block-row i = n / R of
//           sum over c < C of X[t][indices[p] * C + c] * data[p][n - iR][c]      (Sec. 2.2)
// Consecutive threads take consecutive n, so Y stores are coalesced and X reads are broadcasts.
// It is the simplest correct kernel and the fallback for shapes without a tiled kernel.
#include "device_common.h"

namespace bsr {

namespace {

template <bool kBF16>
__device__ __forceinline__ float load_elem(const void *p, int64_t idx) {
    if constexpr (kBF16) {
        return bf16_bits_to_float(static_cast<const unsigned short *>(p)[idx]);
    } else {
        return static_cast<const float *>(p)[idx];
    }
}

template <bool kBF16>
__global__ __launch_bounds__(256) void spmm_generic_kernel(
    const void *__restrict__ X, int64_t T, int64_t ldx, const int32_t *__restrict__ indptr,
    const int32_t *__restrict__ indices, const void *__restrict__ data, int64_t nnzb, int32_t R,
    int32_t C, int64_t N, int64_t Kb, const float *__restrict__ bias, float *__restrict__ Y,
    int64_t ldy) {
    const int64_t total = T * N;
    for (int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x; e < total;
         e += int64_t(gridDim.x) * 256) {
        const int64_t t = e / N, n = e - t * N;
        const int64_t i = n / R, r = n - i * R;
        const int64_t p0 = clamp64(indptr[i], 0, nnzb);
        const int64_t p1 = clamp64(indptr[i + 1], p0, nnzb);
        const int64_t xrow = t * ldx;
        float acc = 0.0f;
        for (int64_t p = p0; p < p1; ++p) {
            const int64_t j = clamp64(indices[p], 0, Kb - 1);
            const int64_t xo = xrow + j * C;
            const int64_t wo = (p * R + r) * C;
            for (int c = 0; c < C; ++c)
                acc = fmaf(load_elem<kBF16>(X, xo + c), load_elem<kBF16>(data, wo + c), acc);
        }
        Y[t * ldy + n] = acc + (bias ? bias[n] : 0.0f);
    }
}

}  // namespace

bsr_status launch_spmm_generic(const void *X, int64_t T, int64_t ldx, const bsr_matrix_t *W,
                               const float *bias, float *Y, int64_t ldy, void *stream,
                               const LaunchEvents &ev) {
    const int64_t N = W->n_rows, Kb = W->n_cols / W->C;
    const dim3 grid(grid_for(T * N, 256)), block(256);
    auto kernel = (W->dtype == BSR_BF16) ? spmm_generic_kernel<true> : spmm_generic_kernel<false>;
    launch_kernel(kernel, grid, block, 0, as_stream(stream), ev, X, T, ldx, W->indptr,
                  W->indices, W->data, W->nnzb, W->R, W->C, N, Kb, bias, Y, ldy);
    return launch_status();
}

}  // namespace bsr
