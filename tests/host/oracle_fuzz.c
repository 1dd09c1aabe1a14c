/* The C oracle (oracle/cpu_oracle.c) on small random BSR matrices, built with AddressSanitizer
 * and UndefinedBehaviorSanitizer by tests/test_host_sanitizers.py: every array is allocated to
 * its exact size, so a read past any of them is reported.  Also checks each product against a
 * plain dense loop on the same data (exact: integer-valued inputs).  Prints "ok". */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

void oracle_block_keys(const float *W, int64_t N, int64_t K, int64_t ldw, int32_t R, int32_t C,
                       double *key);
void oracle_spmm(const float *X, int64_t T, int64_t K, int64_t ldx, const int32_t *indptr,
                 const int32_t *indices, const float *data, int32_t R, int32_t C, int64_t N,
                 const float *bias, double *Y);

static uint64_t s = 88172645463325252ull;
static uint64_t rnd(void) { s ^= s << 13; s ^= s >> 7; s ^= s << 17; return s; }
static float val(void) { return (float)((int)(rnd() % 17) - 8); }

int main(void) {
    const int32_t shapes[] = {1, 2, 3, 4, 8, 16, 32};
    for (int it = 0; it < 3000; ++it) {
        const int32_t R = shapes[rnd() % 7], C = shapes[rnd() % 7];
        const int64_t Nb = 1 + (int64_t)(rnd() % 5), Kb = 1 + (int64_t)(rnd() % 5);
        const int64_t N = Nb * R, K = Kb * C, T = (int64_t)(rnd() % 7);
        const int64_t ldw = K + (int64_t)(rnd() % 3), ldx = K + (int64_t)(rnd() % 3);
        float *W = malloc(sizeof(float) * (size_t)(N * ldw));
        for (int64_t i = 0; i < N * ldw; ++i) W[i] = val();
        double *key = malloc(sizeof(double) * (size_t)(Nb * Kb));
        oracle_block_keys(W, N, K, ldw, R, C, key);
        /* Keep a random subset of blocks, in row order with ascending columns. */
        int32_t *indptr = malloc(sizeof(int32_t) * (size_t)(Nb + 1));
        int32_t *indices = malloc(sizeof(int32_t) * (size_t)(Nb * Kb) + 1);
        float *data = malloc(sizeof(float) * (size_t)(Nb * Kb * R * C) + 1);
        int32_t nnzb = 0;
        indptr[0] = 0;
        for (int64_t i = 0; i < Nb; ++i) {
            for (int64_t j = 0; j < Kb; ++j) {
                if (rnd() % 3 == 0) continue;
                double k2 = 0.0;
                for (int32_t r = 0; r < R; ++r)
                    for (int32_t c = 0; c < C; ++c) {
                        const float x = W[(i * R + r) * ldw + j * C + c];
                        data[((int64_t)nnzb * R + r) * C + c] = x;
                        k2 += (double)x * x;
                    }
                if (k2 != key[i * Kb + j]) { printf("key mismatch\n"); return 1; }
                indices[nnzb++] = (int32_t)j;
            }
            indptr[i + 1] = nnzb;
        }
        float *X = malloc(sizeof(float) * (size_t)(T * ldx) + 1);
        for (int64_t i = 0; i < T * ldx; ++i) X[i] = val();
        float *bias = NULL;
        if (rnd() % 2) {
            bias = malloc(sizeof(float) * (size_t)N);
            for (int64_t i = 0; i < N; ++i) bias[i] = val();
        }
        double *Y = malloc(sizeof(double) * (size_t)(T * N) + 1);
        oracle_spmm(X, T, K, ldx, indptr, indices, data, R, C, N, bias, Y);
        for (int64_t t = 0; t < T; ++t)
            for (int64_t n = 0; n < N; ++n) {
                const int64_t i = n / R, r = n % R;
                double y = bias ? bias[n] : 0.0;
                for (int32_t p = indptr[i]; p < indptr[i + 1]; ++p)
                    for (int32_t c = 0; c < C; ++c)
                        y += (double)X[t * ldx + (int64_t)indices[p] * C + c] *
                             data[((int64_t)p * R + r) * C + c];
                if (y != Y[t * N + n]) { printf("product mismatch\n"); return 1; }
            }
        free(W); free(key); free(indptr); free(indices); free(data); free(X); free(bias); free(Y);
    }
    printf("ok\n");
    return 0;
}
