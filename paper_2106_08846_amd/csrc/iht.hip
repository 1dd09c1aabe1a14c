// The update step of the iterative projection for Eq. 2 (Sec. 2.1): projected gradient descent
// on the layer-output reconstruction loss f(W) = 1/2 tr((W - W0) H (W - W0)^T) under the block
// count bound of Eq. 2, W <- P_k(W - eta (W - W0) H).  The gradient's two products, G = H W^T
// (W the current BSR iterate) and C0 = H W0^T, are BSR products (the symmetric H is their X
// operand); P_k is the block prune.  This kernel joins them:
//   V[n][j] = W[n][j] - eta * (G[j][n] - C0[j][n]),
// each subtraction and the product rounded to fp32 on its own (no fused multiply-add), so the
// result is defined to the bit.  G and C0 are read transposed: a 64 x 64 tile of each goes
// through LDS, read along its rows and written along W's rows.
#include "device_common.h"

namespace bsr {

namespace {

constexpr int kTile = 64;
constexpr int kThreads = 256;

#pragma clang fp contract(off)
__global__ __launch_bounds__(kThreads) void iht_update_kernel(
    const float *__restrict__ W, int64_t ldw, const float *__restrict__ G, int64_t ldg,
    const float *__restrict__ C0, int64_t ldc, float eta, int64_t N, int64_t K, float *V,
    int64_t ldv) {
    __shared__ float sd[kTile][kTile + 1];   // d = G - C0, indexed [j - j0][n - n0]
    const int64_t n0 = int64_t(blockIdx.x) * kTile, j0 = int64_t(blockIdx.y) * kTile;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;   // 64 x 4 threads
    // Rows j of G and C0, columns n: consecutive threads read consecutive n.
    for (int r = ty; r < kTile; r += kThreads / kTile) {
        const int64_t j = j0 + r, n = n0 + tx;
        float d = 0.0f;
        if (j < K && n < N) d = G[j * ldg + n] - C0[j * ldc + n];
        sd[r][tx] = d;
    }
    __syncthreads();
    // Rows n of W and V, columns j: consecutive threads read consecutive j.
    for (int r = ty; r < kTile; r += kThreads / kTile) {
        const int64_t n = n0 + r, j = j0 + tx;
        if (n < N && j < K) {
            const float m = eta * sd[tx][r];
            V[n * ldv + j] = W[n * ldw + j] - m;
        }
    }
}
#pragma clang fp contract(on)

}  // namespace

bsr_status launch_iht_update(const float *W, int64_t ldw, const float *G, int64_t ldg,
                             const float *C0, int64_t ldc, float eta, int64_t N, int64_t K,
                             float *V, int64_t ldv, void *stream) {
    const dim3 grid(unsigned((N + kTile - 1) / kTile), unsigned((K + kTile - 1) / kTile));
    hipLaunchKernelGGL(iht_update_kernel, grid, dim3(kThreads), 0, as_stream(stream), W, ldw, G,
                       ldg, C0, ldc, eta, N, K, V, ldv);
    return launch_status();
}

}  // namespace bsr
