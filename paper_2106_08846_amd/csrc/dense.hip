// BSR -> dense expansion, re-blocking to a finer block shape, and the fp32 -> bf16 cast.
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

// indptr of the re-blocked matrix: fine block-row i*a + r starts at indptr[i]*a*b + r*n*b, with
// n the block count of block-row i.  One thread per fine block-row (plus the final entry).
__global__ __launch_bounds__(256) void reblock_indptr_kernel(const int32_t *__restrict__ indptr,
                                                             int64_t nnzb, int64_t Nb, int32_t a,
                                                             int32_t b, int32_t *__restrict__ out) {
    const int64_t rows = Nb * a;
    for (int64_t i2 = int64_t(blockIdx.x) * 256 + threadIdx.x; i2 <= rows;
         i2 += int64_t(gridDim.x) * 256) {
        int64_t v = nnzb * a * b;
        if (i2 < rows) {
            const int64_t i = i2 / a, r = i2 - i * a;
            const int64_t lo = clamp64(indptr[i], 0, nnzb);
            const int64_t hi = clamp64(indptr[i + 1], lo, nnzb);
            v = lo * a * b + r * (hi - lo) * b;
        }
        out[i2] = int32_t(v);
    }
}

// Indices and values of the re-blocked matrix.  One thread per stored element (block p, row y,
// column x) finds p's block-row by binary search over indptr, then moves the element to piece
// (y / R2, x / C2) of that block; the thread holding a piece's first element writes its column.
// A malformed indptr (a block outside its row's range) drops the element instead of writing
// out of range.
template <typename E>
__global__ __launch_bounds__(256) void reblock_data_kernel(
    const int32_t *__restrict__ indptr, const int32_t *__restrict__ indices,
    const E *__restrict__ data, int64_t nnzb, int64_t Nb, int32_t R, int32_t C, int32_t R2,
    int32_t C2, int32_t *__restrict__ indices_out, E *__restrict__ data_out) {
    const int64_t per = int64_t(R) * C, total = nnzb * per;
    const int32_t a = R / R2, b = C / C2;
    for (int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x; e < total;
         e += int64_t(gridDim.x) * 256) {
        const int64_t p = e / per, rem = e - p * per;
        const int32_t y = int32_t(rem / C), x = int32_t(rem - int64_t(y) * C);
        int64_t lo = 0, hi = Nb;   // last block-row i with indptr[i] <= p
        while (hi - lo > 1) {
            const int64_t mid = (lo + hi) >> 1;
            if (indptr[mid] <= p) lo = mid; else hi = mid;
        }
        const int64_t s0 = clamp64(indptr[lo], 0, nnzb);
        const int64_t s1 = clamp64(indptr[lo + 1], s0, nnzb);
        if (p < s0 || p >= s1) continue;
        const int32_t r = y / R2, yy = y - r * R2, s = x / C2, xx = x - s * C2;
        const int64_t dst = s0 * a * b + int64_t(r) * (s1 - s0) * b + (p - s0) * b + s;
        data_out[(dst * R2 + yy) * C2 + xx] = data[e];
        if (yy == 0 && xx == 0) indices_out[dst] = int32_t(int64_t(indices[p]) * b + s);
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

bsr_status launch_reblock(const bsr_matrix_t *W, int32_t R2, int32_t C2, int32_t *indptr_out,
                          int32_t *indices_out, void *data_out, void *stream) {
    const int64_t Nb = W->n_rows / W->R, nnzb = W->nnzb;
    const int32_t a = W->R / R2, b = W->C / C2;
    const hipStream_t st = as_stream(stream);
    hipLaunchKernelGGL(reblock_indptr_kernel, dim3(grid_for(Nb * a + 1, 256)), dim3(256), 0, st,
                       W->indptr, nnzb, Nb, a, b, indptr_out);
    bsr_status s = launch_status();
    if (s != BSR_OK || nnzb == 0) return s;
    const int64_t total = nnzb * W->R * W->C;
    if (W->dtype == BSR_BF16) {
        hipLaunchKernelGGL(reblock_data_kernel<unsigned short>, dim3(grid_for(total, 256)),
                           dim3(256), 0, st, W->indptr, W->indices,
                           static_cast<const unsigned short *>(W->data), nnzb, Nb, W->R, W->C,
                           R2, C2, indices_out, static_cast<unsigned short *>(data_out));
    } else {
        hipLaunchKernelGGL(reblock_data_kernel<unsigned>, dim3(grid_for(total, 256)), dim3(256),
                           0, st, W->indptr, W->indices, static_cast<const unsigned *>(W->data),
                           nnzb, Nb, W->R, W->C, R2, C2, indices_out,
                           static_cast<unsigned *>(data_out));
    }
    return launch_status();
}

bsr_status launch_cast(const float *src, uint16_t *dst, int64_t n, void *stream) {
    hipLaunchKernelGGL(cast_f32_bf16_kernel, dim3(grid_for(n, 256)), dim3(256), 0,
                       as_stream(stream), reinterpret_cast<const unsigned *>(src),
                       reinterpret_cast<unsigned short *>(dst), n);
    return launch_status();
}

}  // namespace bsr
