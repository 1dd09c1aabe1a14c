// Host-side validation for libbsr's C ABI: pure C++ with no HIP dependency.
//
// Every check here runs before anything is enqueued, so a rejected call launches nothing and
// leaves its outputs untouched.
#include <cmath>
#include <cstdint>
#include <cstring>

#include "bsr_internal.h"

namespace {

constexpr int64_t kMaxBlocks = (int64_t(1) << 31) - 1;   // block ids and indptr are int32
constexpr int64_t kMaxElems = int64_t(1) << 53;          // element offsets stay exact

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

bool tiles(int64_t N, int64_t K, int32_t R, int32_t C) {
    return N > 0 && K > 0 && R > 0 && C > 0 && N % R == 0 && K % C == 0;
}

}  // namespace

namespace bsr {

PruneWorkspace prune_workspace_layout(int64_t nb) {
    PruneWorkspace w{};
    w.key_offset = 0;
    w.key_bytes = size_t(nb) * sizeof(uint64_t);
    w.src_offset = align256(w.key_bytes);
    w.src_bytes = size_t(nb) * sizeof(int32_t);
    w.total = align256(w.src_offset + w.src_bytes);
    return w;
}

bsr_status check_prune(const float *W, int64_t N, int64_t K, int64_t ldw, int32_t R, int32_t C,
                       int64_t k, const int32_t *indptr, const int32_t *indices,
                       const float *data, int64_t capacity_blocks, const void *workspace,
                       size_t ws_bytes) {
    if (!W || !indptr) return BSR_ERR_NULL;
    if (!tiles(N, K, R, C) || ldw < K) return BSR_ERR_SHAPE;
    const int64_t Nb = N / R, Kb = K / C;
    if (Nb > kMaxBlocks / Kb) return BSR_ERR_UNSUPPORTED;
    const int64_t nb = Nb * Kb;
    if (N > kMaxElems / ldw) return BSR_ERR_UNSUPPORTED;
    if (k < 0 || k > nb) return BSR_ERR_ARG;
    if (k > 0 && (!indices || !data)) return BSR_ERR_NULL;
    if (capacity_blocks < k) return BSR_ERR_CAPACITY;
    if (!workspace || ws_bytes < prune_workspace_layout(nb).total) return BSR_ERR_WORKSPACE;
    return BSR_OK;
}

bsr_status check_prune_noalloc(const float *W, int64_t N, int64_t K, int64_t ldw, int32_t R,
                               int32_t C, int64_t k, const int32_t *indptr,
                               const int32_t *indices, const float *data,
                               int64_t capacity_blocks) {
    // The same checks as check_prune, with the library's fixed scratch array standing in for
    // the workspace: a matrix with more blocks than it holds is BSR_ERR_WORKSPACE.
    if (tiles(N, K, R, C)) {
        const int64_t Nb = N / R, Kb = K / C;
        if (Nb <= kMaxBlocks / Kb && Nb * Kb > BSR_NOALLOC_MAX_BLOCKS) {
            const bsr_status s = check_prune(W, N, K, ldw, R, C, k, indptr, indices, data,
                                             capacity_blocks, &kMaxBlocks, 0);
            return s == BSR_OK ? BSR_ERR_WORKSPACE : s;
        }
    }
    return check_prune(W, N, K, ldw, R, C, k, indptr, indices, data, capacity_blocks,
                       &kMaxBlocks, kNoallocScratchBytes);
}

bsr_status check_prune_options(const bsr_prune_options_t *opts, int64_t N, int32_t R,
                               int64_t k) {
    if (!opts) return BSR_OK;
    if (opts->norm != BSR_NORM_L2 && opts->norm != BSR_NORM_L1) return BSR_ERR_ARG;
    if (opts->select != BSR_SELECT_GLOBAL && opts->select != BSR_SELECT_PER_ROW)
        return BSR_ERR_ARG;
    if (opts->select == BSR_SELECT_PER_ROW && k % (N / R) != 0) return BSR_ERR_ARG;
    return BSR_OK;
}

bsr_status check_matrix(const bsr_matrix_t *W) {
    if (!W) return BSR_ERR_NULL;
    const int32_t dt = raw_enum(W->dtype);
    if (dt != BSR_F32 && dt != BSR_BF16) return BSR_ERR_ARG;
    if (!tiles(W->n_rows, W->n_cols, W->R, W->C)) return BSR_ERR_SHAPE;
    const int64_t Nb = W->n_rows / W->R, Kb = W->n_cols / W->C;
    if (Nb > kMaxBlocks / Kb) return BSR_ERR_UNSUPPORTED;
    if (W->nnzb < 0 || W->nnzb > Nb * Kb) return BSR_ERR_ARG;
    if (int64_t(W->R) * W->C > kMaxElems / (W->nnzb > 0 ? W->nnzb : 1))
        return BSR_ERR_UNSUPPORTED;
    if (!W->indptr) return BSR_ERR_NULL;
    if (W->nnzb > 0 && (!W->indices || !W->data)) return BSR_ERR_NULL;
    return BSR_OK;
}

namespace {

// Whether the byte ranges [a, a + na) and [b, b + nb) intersect (empty ranges never do).
bool overlaps(const void *a, int64_t na, const void *b, int64_t nb) {
    if (!a || !b || na <= 0 || nb <= 0) return false;
    const uintptr_t pa = reinterpret_cast<uintptr_t>(a), pb = reinterpret_cast<uintptr_t>(b);
    return pa < pb + uint64_t(nb) && pb < pa + uint64_t(na);
}

// Bytes spanned by the arrays of a valid matrix.
int64_t indptr_bytes(const bsr_matrix_t *W) { return (W->n_rows / W->R + 1) * 4; }
int64_t data_bytes(const bsr_matrix_t *W) {
    return W->nnzb * W->R * W->C * (W->dtype == BSR_BF16 ? 2 : 4);
}

}  // namespace

bsr_status check_spmm(const void *X, int x_dtype, int64_t T, int64_t ldx, const bsr_matrix_t *W,
                      const float *Y, int64_t ldy, const float *bias) {
    if (!W) return BSR_ERR_NULL;
    bsr_status s = check_matrix(W);
    if (s != BSR_OK) return s;
    if (x_dtype != BSR_F32 && x_dtype != BSR_BF16) return BSR_ERR_ARG;
    if (x_dtype != int(W->dtype)) return BSR_ERR_DTYPE;
    if (T < 0 || ldx < W->n_cols || ldy < W->n_rows) return BSR_ERR_SHAPE;
    if (T > 0 && (!X || !Y)) return BSR_ERR_NULL;
    if (T > kMaxElems / ldx || T > kMaxElems / ldy) return BSR_ERR_UNSUPPORTED;
    if (T > 0) {
        // Y must not overlap the product's inputs.
        const int64_t yb = ((T - 1) * ldy + W->n_rows) * 4;
        const int64_t xb = ((T - 1) * ldx + W->n_cols) * (x_dtype == BSR_BF16 ? 2 : 4);
        if (overlaps(Y, yb, X, xb) || overlaps(Y, yb, bias, W->n_rows * 4) ||
            overlaps(Y, yb, W->indptr, indptr_bytes(W)) ||
            overlaps(Y, yb, W->indices, W->nnzb * 4) || overlaps(Y, yb, W->data, data_bytes(W)))
            return BSR_ERR_ARG;
    }
    return BSR_OK;
}

bsr_status check_spmm_items(const bsr_spmm_item_t *items, int32_t n) {
    // Products of one call may run concurrently: each Y must be disjoint from every other
    // product's inputs and output (inputs may be shared).  Items are already checked one by
    // one, so every descriptor is valid here.
    auto y_bytes = [](const bsr_spmm_item_t &it) { return ((it.T - 1) * it.ldy + it.W->n_rows) * 4; };
    for (int32_t i = 0; i < n; ++i) {
        const bsr_spmm_item_t &a = items[i];
        if (a.T <= 0) continue;
        const int64_t yb = y_bytes(a);
        for (int32_t j = 0; j < n; ++j) {
            const bsr_spmm_item_t &b = items[j];
            if (j == i || b.T <= 0) continue;
            const bsr_matrix_t *W = b.W;
            const int64_t xb = ((b.T - 1) * b.ldx + W->n_cols) * (b.x_dtype == BSR_BF16 ? 2 : 4);
            if (overlaps(a.Y, yb, b.X, xb) || overlaps(a.Y, yb, b.bias, W->n_rows * 4) ||
                overlaps(a.Y, yb, W->indptr, indptr_bytes(W)) ||
                overlaps(a.Y, yb, W->indices, W->nnzb * 4) ||
                overlaps(a.Y, yb, W->data, data_bytes(W)) || overlaps(a.Y, yb, b.Y, y_bytes(b)))
                return BSR_ERR_ARG;
        }
    }
    return BSR_OK;
}

bsr_status check_plan_use(const bsr_spmm_item_t &it, const bsr_plan_t *plan,
                          int64_t layout_bytes) {
    // The plan must describe this product's matrix (the same arrays and shape) and fit its
    // recorded layout; its memory must not overlap the product's output.
    const bsr_matrix_t *W = it.W;
    if (!plan->mem) return BSR_ERR_NULL;
    if (plan->n_rows != W->n_rows || plan->n_cols != W->n_cols || plan->nnzb != W->nnzb ||
        plan->R != W->R || plan->C != W->C || plan->dtype != int(W->dtype) ||
        plan->indptr != W->indptr || plan->indices != W->indices || plan->data != W->data)
        return BSR_ERR_ARG;
    if (layout_bytes <= 0 || int64_t(plan->bytes) < layout_bytes) return BSR_ERR_ARG;
    if (it.T > 0 && overlaps(it.Y, ((it.T - 1) * it.ldy + W->n_rows) * 4, plan->mem,
                             int64_t(plan->bytes)))
        return BSR_ERR_ARG;
    return BSR_OK;
}

bsr_status check_plan_prepare(const bsr_matrix_t *W, const void *mem, size_t bytes,
                              int64_t layout_bytes) {
    // mem must hold the layout and not overlap the matrix it reads.
    if (!mem) return BSR_ERR_NULL;
    if (int64_t(bytes) < layout_bytes) return BSR_ERR_WORKSPACE;
    if (overlaps(mem, layout_bytes, W->indptr, indptr_bytes(W)) ||
        overlaps(mem, layout_bytes, W->indices, W->nnzb * 4) ||
        overlaps(mem, layout_bytes, W->data, data_bytes(W)))
        return BSR_ERR_ARG;
    return BSR_OK;
}

bsr_status check_to_dense(const bsr_matrix_t *W, const float *out, int64_t ldo) {
    if (!W || !out) return BSR_ERR_NULL;
    bsr_status s = check_matrix(W);
    if (s != BSR_OK) return s;
    if (W->dtype != BSR_F32) return BSR_ERR_DTYPE;
    if (ldo < W->n_cols) return BSR_ERR_SHAPE;
    if (W->n_rows > kMaxElems / ldo) return BSR_ERR_UNSUPPORTED;
    return BSR_OK;
}

bsr_status check_reblock(const bsr_matrix_t *W, int32_t R2, int32_t C2,
                         const int32_t *indptr_out, const int32_t *indices_out,
                         const void *data_out) {
    bsr_status s = check_matrix(W);
    if (s != BSR_OK) return s;
    if (R2 <= 0 || C2 <= 0 || W->R % R2 != 0 || W->C % C2 != 0) return BSR_ERR_SHAPE;
    if (!indptr_out) return BSR_ERR_NULL;
    if (W->nnzb > 0 && (!indices_out || !data_out)) return BSR_ERR_NULL;
    const int64_t pieces = int64_t(W->R / R2) * (W->C / C2);
    const int64_t Nb = W->n_rows / R2, Kb = W->n_cols / C2;
    if (Nb > kMaxBlocks / Kb) return BSR_ERR_UNSUPPORTED;
    if (W->nnzb > kMaxBlocks / pieces) return BSR_ERR_UNSUPPORTED;
    // Outputs must not overlap the inputs or each other.
    const int64_t n2 = W->nnzb * pieces;
    const int64_t outs[3] = {(Nb + 1) * 4, n2 * 4, data_bytes(W)};
    const void *optr[3] = {indptr_out, indices_out, data_out};
    const void *iptr[3] = {W->indptr, W->indices, W->data};
    const int64_t ins[3] = {indptr_bytes(W), W->nnzb * 4, data_bytes(W)};
    for (int i = 0; i < 3; ++i) {
        for (int j = 0; j < 3; ++j)
            if (overlaps(optr[i], outs[i], iptr[j], ins[j])) return BSR_ERR_ARG;
        for (int j = i + 1; j < 3; ++j)
            if (overlaps(optr[i], outs[i], optr[j], outs[j])) return BSR_ERR_ARG;
    }
    return BSR_OK;
}

bsr_status check_cast(const float *src, const uint16_t *dst, int64_t n) {
    if (n < 0) return BSR_ERR_SHAPE;
    if (n > 0 && (!src || !dst)) return BSR_ERR_NULL;
    if (n > kMaxElems) return BSR_ERR_UNSUPPORTED;
    return BSR_OK;
}

bsr_status check_iht_update(const float *W, int64_t ldw, const float *G, int64_t ldg,
                            const float *C0, int64_t ldc, float eta, int64_t N, int64_t K,
                            const float *V, int64_t ldv) {
    if (N < 0 || K < 0) return BSR_ERR_SHAPE;
    if (ldw < K || ldv < K || ldg < N || ldc < N) return BSR_ERR_SHAPE;
    if (!std::isfinite(eta)) return BSR_ERR_ARG;
    if (N == 0 || K == 0) return BSR_OK;
    if (!W || !G || !C0 || !V) return BSR_ERR_NULL;
    if (N > kMaxElems / ldw || N > kMaxElems / ldv || K > kMaxElems / ldg ||
        K > kMaxElems / ldc || N > (int64_t(1) << 37) || K > int64_t(65535) * 64)
        return BSR_ERR_UNSUPPORTED;
    // V may be W itself (each element is read before it is written, by the same thread), but
    // no other overlap of V with an input.
    const int64_t vb = ((N - 1) * ldv + K) * 4;
    if (overlaps(V, vb, G, ((K - 1) * ldg + N) * 4) || overlaps(V, vb, C0, ((K - 1) * ldc + N) * 4))
        return BSR_ERR_ARG;
    if (V != W && overlaps(V, vb, W, ((N - 1) * ldw + K) * 4)) return BSR_ERR_ARG;
    if (V == W && ldv != ldw) return BSR_ERR_ARG;
    return BSR_OK;
}

bsr_status check_attention(const float *Q, int64_t ldq, const float *K, int64_t ldk,
                           const float *V, int64_t ldv, const float *O, int64_t ldo,
                           int32_t batch, int32_t seq, int32_t heads, int32_t head_dim,
                           float scale) {
    if (batch < 0 || seq < 0 || heads < 1 || head_dim < 1) return BSR_ERR_SHAPE;
    const int64_t width = int64_t(heads) * head_dim;
    if (ldq < width || ldk < width || ldv < width || ldo < width) return BSR_ERR_SHAPE;
    if (!std::isfinite(scale)) return BSR_ERR_ARG;
    if (int64_t(batch) * seq == 0) return BSR_OK;
    if (!Q || !K || !V || !O) return BSR_ERR_NULL;
    if (head_dim != 64 || batch > 65535 || heads > 65535) return BSR_ERR_UNSUPPORTED;
    auto aligned = [](const void *p, int64_t ld) {
        return (reinterpret_cast<uintptr_t>(p) & 15) == 0 && ld % 4 == 0;
    };
    if (!aligned(Q, ldq) || !aligned(K, ldk) || !aligned(V, ldv)) return BSR_ERR_UNSUPPORTED;
    const int64_t T = int64_t(batch) * seq;
    if (T > kMaxElems / ldq || T > kMaxElems / ldk || T > kMaxElems / ldv || T > kMaxElems / ldo)
        return BSR_ERR_UNSUPPORTED;
    return BSR_OK;
}

}  // namespace bsr

extern "C" {

bsr_status bsr_prune_count(int64_t N, int64_t K, int32_t R, int32_t C, double density,
                           int64_t *k) {
    if (!k) return BSR_ERR_NULL;
    if (!tiles(N, K, R, C)) return BSR_ERR_SHAPE;
    if (!(density >= 0.0 && density <= 1.0)) return BSR_ERR_ARG;  // rejects NaN too
    const int64_t Nb = N / R, Kb = K / C;
    if (Nb > kMaxBlocks / Kb) return BSR_ERR_UNSUPPORTED;
    const int64_t nb = Nb * Kb;
    double v = std::floor(density * double(nb) + 0.5);
    int64_t kk = int64_t(v);
    if (kk < 0) kk = 0;
    if (kk > nb) kk = nb;
    *k = kk;
    return BSR_OK;
}

bsr_status bsr_prune_count_ex(int64_t N, int64_t K, int32_t R, int32_t C, double density,
                              const bsr_prune_options_t *opts, int64_t *k) {
    const int32_t norm = opts ? opts->norm : BSR_NORM_L2;
    const int32_t select = opts ? opts->select : BSR_SELECT_GLOBAL;
    if (norm != BSR_NORM_L2 && norm != BSR_NORM_L1) return BSR_ERR_ARG;
    if (select != BSR_SELECT_GLOBAL && select != BSR_SELECT_PER_ROW) return BSR_ERR_ARG;
    if (select == BSR_SELECT_GLOBAL) return bsr_prune_count(N, K, R, C, density, k);
    if (!k) return BSR_ERR_NULL;
    if (!tiles(N, K, R, C)) return BSR_ERR_SHAPE;
    if (!(density >= 0.0 && density <= 1.0)) return BSR_ERR_ARG;
    const int64_t Nb = N / R, Kb = K / C;
    if (Nb > kMaxBlocks / Kb) return BSR_ERR_UNSUPPORTED;
    int64_t kr = int64_t(std::floor(density * double(Kb) + 0.5));
    if (kr < 0) kr = 0;
    if (kr > Kb) kr = Kb;
    *k = Nb * kr;
    return BSR_OK;
}

size_t bsr_prune_workspace_bytes(int64_t N, int64_t K, int32_t R, int32_t C) {
    if (!tiles(N, K, R, C)) return 0;
    const int64_t Nb = N / R, Kb = K / C;
    if (Nb > kMaxBlocks / Kb) return 0;
    return bsr::prune_workspace_layout(Nb * Kb).total;
}

const char *bsr_status_str(bsr_status s) {
    switch (s) {
        case BSR_OK: return "ok";
        case BSR_ERR_NULL: return "null pointer argument";
        case BSR_ERR_SHAPE: return "invalid shape or leading dimension";
        case BSR_ERR_ARG: return "invalid argument value";
        case BSR_ERR_DTYPE: return "dtype mismatch";
        case BSR_ERR_CAPACITY: return "output capacity too small";
        case BSR_ERR_WORKSPACE: return "workspace missing or too small";
        case BSR_ERR_HIP: return "HIP runtime error";
        case BSR_ERR_ARCH: return "device is not gfx950";
        case BSR_ERR_UNSUPPORTED: return "unsupported size";
    }
    return "unknown status";
}

}  // extern "C"
