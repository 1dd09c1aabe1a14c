// Internal declarations shared by libbsr's translation units (not part of the C ABI).
#pragma once

#include <stddef.h>
#include <stdint.h>
#include <string.h>

#include "../../include/libbsr.h"

namespace bsr {

// The integer in an enum-typed field or argument a caller passed (a C caller may store any
// int32 there), read as bytes: loading an enum lvalue that names no enumerator is undefined in
// C++, so validation reads enums this way before checking them.
template <class E>
inline int32_t raw_enum(const E &e) {
    static_assert(sizeof(E) == sizeof(int32_t), "the ABI's enums are 32-bit");
    int32_t v;
    memcpy(&v, &e, sizeof v);
    return v;
}

// Workspace layout of the pruning pipeline: fp64 key bits per block, then the source block id
// of every kept block.  Each region starts on a 256-byte boundary.
struct PruneWorkspace {
    size_t key_offset, key_bytes;
    size_t src_offset, src_bytes;
    size_t total;
};
PruneWorkspace prune_workspace_layout(int64_t nb);

// Host-side argument checks; pure C++ (no HIP), so they also run where no GPU exists.
bsr_status check_prune(const float *W, int64_t N, int64_t K, int64_t ldw, int32_t R, int32_t C,
                       int64_t k, const int32_t *indptr, const int32_t *indices,
                       const float *data, int64_t capacity_blocks, const void *workspace,
                       size_t ws_bytes);
// bsr_prune_from_dense_noalloc: the workspace lives in a fixed device array of this many bytes,
// the prune workspace of BSR_NOALLOC_MAX_BLOCKS blocks (8-byte keys, then 4-byte source ids,
// each region a multiple of 256 bytes).
constexpr size_t kNoallocScratchBytes = size_t(BSR_NOALLOC_MAX_BLOCKS) * 8 +
                                        size_t(BSR_NOALLOC_MAX_BLOCKS) * 4;
static_assert(BSR_NOALLOC_MAX_BLOCKS % 64 == 0, "both regions stay 256-byte multiples");
bsr_status check_prune_noalloc(const float *W, int64_t N, int64_t K, int64_t ldw, int32_t R,
                               int32_t C, int64_t k, const int32_t *indptr,
                               const int32_t *indices, const float *data,
                               int64_t capacity_blocks);
// Device address of this device's scratch array (found once per device, with it current).
bsr_status noalloc_scratch(void **ptr);
// Options of the _ex pruning entry point (after check_prune: N, R valid, k in [0, nb]).
bsr_status check_prune_options(const bsr_prune_options_t *opts, int64_t N, int32_t R, int64_t k);
bsr_status check_matrix(const bsr_matrix_t *W);
bsr_status check_spmm(const void *X, int x_dtype, int64_t T, int64_t ldx, const bsr_matrix_t *W,
                      const float *Y, int64_t ldy, const float *bias);
// A plan used by a product (after check_spmm): it describes the item's matrix, its recorded
// size covers `layout_bytes`, and it does not overlap the item's Y.
bsr_status check_plan_use(const bsr_spmm_item_t &it, const bsr_plan_t *plan,
                          int64_t layout_bytes);
// Plan memory for a matrix (after check_matrix): large enough, not overlapping the matrix.
bsr_status check_plan_prepare(const bsr_matrix_t *W, const void *mem, size_t bytes,
                              int64_t layout_bytes);
// Cross-product aliasing of a batched call (after check_spmm on every item).
bsr_status check_spmm_items(const bsr_spmm_item_t *items, int32_t n);
bsr_status check_to_dense(const bsr_matrix_t *W, const float *out, int64_t ldo);
bsr_status check_cast(const float *src, const uint16_t *dst, int64_t n);
bsr_status check_iht_update(const float *W, int64_t ldw, const float *G, int64_t ldg,
                            const float *C0, int64_t ldc, float eta, int64_t N, int64_t K,
                            const float *V, int64_t ldv);
bsr_status check_reblock(const bsr_matrix_t *W, int32_t R2, int32_t C2,
                         const int32_t *indptr_out, const int32_t *indices_out,
                         const void *data_out);
bsr_status check_attention(const float *Q, int64_t ldq, const float *K, int64_t ldk,
                           const float *V, int64_t ldv, const float *O, int64_t ldo,
                           int32_t batch, int32_t seq, int32_t heads, int32_t head_dim,
                           float scale);

// Device-side entry points (implemented in the .hip files).  Arguments are already validated.
bsr_status ensure_device();  // current device is gfx950; caches its properties
int device_cu_count();
int auto_slices(const int64_t *tiles, int n, int cu_count);  // token tiles per product
size_t device_lds_per_block();

bsr_status launch_prune(const float *W, int64_t N, int64_t K, int64_t ldw, int32_t R, int32_t C,
                        int64_t k, int32_t *indptr, int32_t *indices, float *data,
                        void *workspace, int norm, int select, void *stream);
bsr_status launch_to_dense(const bsr_matrix_t *W, float *out, int64_t ldo, void *stream);
bsr_status launch_cast(const float *src, uint16_t *dst, int64_t n, void *stream);
bsr_status launch_iht_update(const float *W, int64_t ldw, const float *G, int64_t ldg,
                             const float *C0, int64_t ldc, float eta, int64_t N, int64_t K,
                             float *V, int64_t ldv, void *stream);
bsr_status launch_reblock(const bsr_matrix_t *W, int32_t R2, int32_t C2, int32_t *indptr_out,
                          int32_t *indices_out, void *data_out, void *stream);
// Optional event pair recorded at a product kernel's start and end (hipExtLaunchKernel).
struct LaunchEvents {
    void *start = nullptr;
    void *stop = nullptr;
};

bsr_status launch_spmm_generic(const void *X, int64_t T, int64_t ldx, const bsr_matrix_t *W,
                               const float *bias, float *Y, int64_t ldy, void *stream,
                               const LaunchEvents &ev);

bsr_status launch_attention(const float *Q, int64_t ldq, const float *K, int64_t ldk,
                            const float *V, int64_t ldv, float *O, int64_t ldo, int batch,
                            int seq, int heads, float scale, void *stream);

void set_last_hip_error(const char *msg);

}  // namespace bsr
