// Launch planning for the LDS-tiled BSR product kernels (matrix-core and vector-ALU).
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "bsr_internal.h"

namespace bsr {

struct TiledPlan {
    bool ok = false;
    int tokens = 32;        // tokens per tile: 32, or 64 (bf16 32x1 blocks, many tokens)
    int num_tiles = 0;      // token tiles
    int slices = 1;         // block-row slices per token tile
    int x_pitch = 0;        // LDS row pitch of the X tile, in floats
    int indptr_words = 0;   // LDS words reserved for indptr
    int bias_words = 0;     // LDS words reserved for the bias
    int wbuf_offset = 0;    // bytes from the X tile to the per-wave block scratch (if any)
    int ib_offset = 0;      // R x 1 kernels: LDS words from the unit row pointer to indptr
    size_t lds_bytes = 0;   // dynamic LDS per workgroup
};

// Whether a tiled kernel exists for this block shape and dtype.
bool tiled_supported(int R, int C, int dtype);
int tiled_waves(int R, int C);  // waves per workgroup

// Row pitch, in elements, of a row-major X tile of `cols` columns for the matrix-core units.
// The pitch decides which LDS banks the units' operand reads hit; these rules were measured
// with SQ_LDS_BANK_CONFLICT on MI355X (gfx950):
//  * 32x1 (ds_read_b32 gathers; a half-wave reads 32 tokens of one column): an odd pitch.
//  * 16x1 (a half-wave reads 16 tokens of each of two columns): pitch = 2 (mod 32); two
//    columns an odd distance apart then hit disjoint banks (an even distance still conflicts:
//    with 32 banks no pitch separates every pair).
//  * 32x32 fp32 (ds_read_b128; lane l reads token l % 32, quad l / 32): pitch = 4 (mod 8).
//  * 16x16 fp32 (ds_read_b128; lane l reads token l % 16, quad l / 16): pitch = 8 (mod 16).
//  * bf16 square tiles (ds_read_b64 of bf16 pairs): cols + 8 bf16.
// The R x 1 tiles also hold a zero column at index `cols`, so their pitch is at least cols + 1.
inline int64_t tile_pitch(int R, int C, bool tile_bf16, int64_t cols) {
    if (C == 1) {
        if (R == 16) return cols + 1 + (((1 - cols) % 32) + 32) % 32;
        return cols + ((cols & 1) ? 2 : 1);
    }
    if (tile_bf16) return cols + 8;
    return R == 16 ? cols + 8 : cols + 4;   // cols is a multiple of C
}

// Plan a tiled launch; plan.ok is false when the shape does not fit (LDS, alignment, sizes).
// slices <= 0 leaves the slice count at 1; the caller picks it.
TiledPlan plan_tiled(const void *X, int64_t T, int64_t ldx, const bsr_matrix_t *W, int64_t ldy,
                     int slices, size_t lds_limit);

// Most products one tiled launch takes (all with the same block shape and dtype).
constexpr int kMaxItems = 8;

// One product of a tiled launch, as planned on the host (plan_mem and the offsets: the
// product's per-matrix plan, or NULL).
struct TiledWork {
    TiledPlan plan;
    const void *X;
    int64_t T, ldx;
    const bsr_matrix_t *W;
    const float *bias;
    float *Y;
    int64_t ldy;
    const void *plan_mem = nullptr;
    int64_t plan_uptr_offset = 0, plan_col_offset = 0, plan_val_offset = 0, plan_max_units = 0;
    int plan_arith = 0;   // with a plan: BSR_ARITH_NATIVE or BSR_ARITH_BF16X3
};

// The device-side view of one product, passed by value in the kernel arguments.
struct TiledItem {
    const void *X;
    int64_t T, ldx;
    const int32_t *indptr;
    const int32_t *indices;
    const void *data;   // fp32 or bf16 blocks
    const float *bias;
    float *Y;
    int64_t ldy;
    int K, nnzb, Nb, Kb;
    int num_tiles, slices, XP, indptr_words, bias_words, wbuf_offset;
    // R x 1 kernels: LDS words from the unit row pointer to indptr; with a plan, its unit row
    // pointer, packed columns and weights, and its reserved units.
    int ib_offset, ucap;
    const int32_t *uptr;
    const int32_t *ucol;
    const void *uval;
    // Planned flat launches of paired products (see launch_spmm_flat): the batch index of the
    // product that shares this one's workgroups and X tiles, or -1.
    int partner;
};

struct TiledBatch {
    int n;
    TiledItem item[kMaxItems];
};

// bf16 32x1 products take 64-token tiles when their block-rows hold at least this many stored
// blocks on average (measured on MI355X, fused QKV 2304x768 at 4096 tokens: 12% faster at 307
// blocks per row, 1% at 154, 3% slower at 77 and 5% slower at 38).
constexpr int64_t kTile64RowBlocks = 128;

// 16x16 launches use four-block units when the products' block-rows hold at least this many
// stored blocks on average (measured on MI355X: faster from about 8, slower below).
constexpr int kWideUnitRowBlocks = 8;
bool wide_units(const TiledWork *work, int n);

// Launch 1..kMaxItems planned products of one block shape as a single kernel.
bsr_status launch_spmm_tiled(const TiledWork *work, int n, void *stream, const LaunchEvents &ev);

// The flat-stream kernel for linear R x 1 blocks (32x1, 16x1): same plan and batch structures
// as the tiled kernel; `planned` launches read per-matrix plans (32x1 only), and every product
// of one launch has a plan of the same arithmetic or none has.
bool flat_supported(int R, int C, int dtype);
// The resolved arithmetic of a plan request (BSR_ARITH_AUTO -> BSR_ARITH_NATIVE), or -1 for a
// value that names no arithmetic.
int resolve_arith(int dtype, int arith);
// Whether a plan of this arithmetic exists for the block shape and dtype.
bool plan_supported(int R, int C, int dtype, int arith);
int flat_unit_blocks(int R, int C, int dtype);   // blocks per unit (0 if unsupported)
bsr_status launch_spmm_flat(const TiledWork *work, int n, bool planned, void *stream,
                            const LaunchEvents &ev);

// Per-matrix plans: layout and the preparing kernels (plan.hip).
struct PlanLayout {
    int unit_blocks = 0;
    int arith = 0;   // resolved
    int64_t max_units = 0;
    int64_t uptr_offset = 0, col_offset = 0, val_offset = 0, total = 0;
};
PlanLayout plan_layout(const bsr_matrix_t *W, int arith);   // unit_blocks = 0 when unsupported
bsr_status launch_plan_prepare(const bsr_matrix_t *W, void *mem, const PlanLayout &L,
                               void *stream);

// The column-chunked matrix-core kernel, for inputs too wide for one LDS X tile: same units
// and shapes as the tiled kernel; the plan also fills chunk_blocks and nchunks.
struct KchunkPlan {
    TiledPlan base;
    int chunk_blocks = 0;   // block-columns per chunk (the last chunk may be narrower)
    int nchunks = 0;
};
KchunkPlan plan_kchunk(const void *X, int64_t T, int64_t ldx, const bsr_matrix_t *W,
                       int64_t ldy, int slices, size_t lds_limit);

struct KchunkItem {
    const void *X;
    int64_t T, ldx;
    const int32_t *indptr;
    const int32_t *indices;
    const void *data;
    const float *bias;
    float *Y;
    int64_t ldy;
    int nnzb, Nb, Kb;
    int num_tiles, slices, XP, bias_words, wbuf_offset, chunk_blocks, nchunks;
};

struct KchunkBatch {
    int n;
    KchunkItem item[kMaxItems];
};

struct KchunkWork {
    KchunkPlan plan;
    const void *X;
    int64_t T, ldx;
    const bsr_matrix_t *W;
    const float *bias;
    float *Y;
    int64_t ldy;
};
bsr_status launch_spmm_kchunk(const KchunkWork *work, int n, void *stream,
                              const LaunchEvents &ev);

// The vector-ALU tile kernel (shapes without a matrix-core kernel: 1 x C, 2x1 .. 8x1, 2x2 ..
// 8x8).  Same plan and batch structures; the plan fills num_tiles, slices, x_pitch, lds_bytes.
bool vtile_supported(int R, int C, int dtype);
TiledPlan plan_vtile(const void *X, int64_t T, int64_t ldx, const bsr_matrix_t *W, int64_t ldy,
                     int slices, size_t lds_limit);
bsr_status launch_spmm_vtile(const TiledWork *work, int n, void *stream, const LaunchEvents &ev);

// The column-chunked vector-ALU kernel, for the same shapes when the X tile does not fit.
KchunkPlan plan_vchunk(const void *X, int64_t T, int64_t ldx, const bsr_matrix_t *W,
                       int64_t ldy, int slices, size_t lds_limit);
bsr_status launch_spmm_vchunk(const KchunkWork *work, int n, void *stream,
                              const LaunchEvents &ev);

}  // namespace bsr
