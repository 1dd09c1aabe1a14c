/*
 * Plain C oracle for BSR pruning keys and BSR x dense products, fp64 accumulation.
 *
 * TEST INFRASTRUCTURE ONLY: loaded by the test suite and by the CPU-baseline timing leg of the
 * benchmark.  It shares no source with the GPU library and is checked against the numpy oracle.
 *
 * Definitions followed:
 *  - Sec. 2.1, Eq. 3 with the l2 group norm: key(i, j) = sum over the R x C block of w^2, summed
 *    in fp64, row r outer, column c inner, from +0.0.
 *  - Sec. 2.2 (BSR as data / indices / indptr, SciPy layout; only stored blocks are multiplied):
 *    Y[t][n] = b[n] + sum over stored blocks p of block-row i = n / R, sum over c < C of
 *    X[t][indices[p] * C + c] * data[p][n - i R][c].
 *
 * Threads: the token loop is split over OpenMP threads; each output element is still one plain
 * sequential fp64 sum.
 */
#include <stdint.h>
#include <stddef.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Number of OpenMP threads a parallel region will use (1 without OpenMP). */
int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Set the OpenMP thread count for later calls (ignored without OpenMP). */
void oracle_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* key[i * Kb + j] for every R x C block of the row-major N x K fp32 matrix W (row pitch ldw). */
void oracle_block_keys(const float *W, int64_t N, int64_t K, int64_t ldw, int32_t R, int32_t C,
                       double *key)
{
    int64_t Nb = N / R, Kb = K / C;
    for (int64_t i = 0; i < Nb; ++i) {
        for (int64_t j = 0; j < Kb; ++j) {
            double s = 0.0;
            for (int32_t r = 0; r < R; ++r) {
                for (int32_t c = 0; c < C; ++c) {
                    double x = (double)W[(i * R + r) * ldw + j * C + c];
                    s = s + x * x;
                }
            }
            key[i * Kb + j] = s;
        }
    }
}

/*
 * Y (T x N, fp64, row pitch N) = X (T x K, fp32, row pitch ldx) times the transpose of the BSR
 * matrix (indptr[N/R + 1], indices[nnzb], data[nnzb][R][C] fp32), plus bias (nullable, [N]).
 */
void oracle_spmm(const float *X, int64_t T, int64_t K, int64_t ldx,
                 const int32_t *indptr, const int32_t *indices, const float *data,
                 int32_t R, int32_t C, int64_t N, const float *bias, double *Y)
{
    int64_t Nb = N / R;
    (void)K;
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < T; ++t) {
        const float *x = X + t * ldx;
        double *y = Y + t * N;
        for (int64_t i = 0; i < Nb; ++i) {
            for (int32_t r = 0; r < R; ++r) {
                double s = bias ? (double)bias[i * R + r] : 0.0;
                for (int32_t p = indptr[i]; p < indptr[i + 1]; ++p) {
                    const float *blk = data + ((int64_t)p * R + r) * C;
                    const float *xs = x + (int64_t)indices[p] * C;
                    for (int32_t c = 0; c < C; ++c)
                        s = s + (double)xs[c] * (double)blk[c];
                }
                y[i * R + r] = s;
            }
        }
    }
}
