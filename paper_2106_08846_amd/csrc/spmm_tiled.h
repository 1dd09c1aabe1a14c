// Launch planning for the tiled (MFMA) BSR product kernels.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "bsr_internal.h"

namespace bsr {

struct TiledPlan {
    bool ok = false;
    int num_tiles = 0;      // 32-token tiles
    int slices = 1;         // block-row slices per token tile
    int x_pitch = 0;        // LDS row pitch of the X tile, in floats
    int indptr_words = 0;   // LDS words reserved for indptr
    int x_vec4 = 0;         // X rows can be read as float4
    size_t lds_bytes = 0;   // dynamic LDS per workgroup
};

// Whether a tiled kernel exists for this block shape and dtype.
bool tiled_supported(int R, int C, int dtype);
int tiled_waves(int R, int C);  // waves per workgroup

// Plan a tiled launch; plan.ok is false when the shape does not fit (LDS, alignment, sizes).
// slices <= 0 leaves the slice count at 1; the caller picks it.
TiledPlan plan_tiled(const void *X, int64_t T, int64_t ldx, const bsr_matrix_t *W, int slices,
                     size_t lds_limit);

bsr_status launch_spmm_tiled(const TiledPlan &plan, const void *X, int64_t T, int64_t ldx,
                             const bsr_matrix_t *W, const float *bias, float *Y, int64_t ldy,
                             void *stream);

}  // namespace bsr
