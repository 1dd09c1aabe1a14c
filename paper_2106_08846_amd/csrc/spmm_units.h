// Matrix-core "units" of the BSR product kernels (fp32 accumulate): per block shape and input
// type, how a wave loads a group of stored blocks (a unit) into registers, runs its MFMAs
// against an X tile in LDS, and stores a finished 32-token tile of Y.
//
//   * R x 1 blocks (32x1, 16x1): the contraction index is the block.  32x1 uses
//     v_mfma_f32_32x32x2_f32 with two blocks per instruction; lane l supplies token l%32 of
//     block l/32 (gathered from the LDS X tile) and feature l%32 of that block's data, so the B
//     operand is one contiguous 256-byte load per instruction.  16x1 uses
//     v_mfma_f32_16x16x4_f32, four blocks per instruction, for two 16-token halves.  32x1 bf16
//     uses v_mfma_f32_32x32x16_bf16 on a transposed bf16 tile.
//   * R x R blocks (32x32, 16x16): the contraction index is the block column c.  Each lane
//     loads 16 contiguous bytes of the block (one float4 of a block row), and the order of c
//     inside each instruction is permuted identically for the A and B operands, which the sum
//     does not see.  A comes from the LDS X tile with 16-byte reads.
//
// Every unit offers: zero / init (bias) / load / mask (partial unit) / mma / store / store_reg /
// get / add, plus its tile layout (kPad: the smallest pitch padding, 1 for the R x 1 tiles with
// their zero column; kTileBF16, kTransposed) and blocks per unit (KB).  The planner's
// tile_pitch() sets the pitch itself.
// Column indices are relative to the X tile; lanes with index -1 read the tile's zero column.
#pragma once

#include <type_traits>

#include "device_common.h"

namespace bsr {

namespace {
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef short shortx4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned uintx4 __attribute__((ext_vector_type(4)));
typedef unsigned uintx2 __attribute__((ext_vector_type(2)));
typedef unsigned short bf16_t;  // a bf16 value as its bit pattern
typedef short shortx8 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) shortx4 lds_shortx4;

constexpr int kTT = 32;           // tokens per workgroup
constexpr int kStageChunks = 12;  // 64-column chunks of an X row in flight per wave

__device__ __forceinline__ floatx16 mfma32(float a, float b, floatx16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ floatx4 mfma16(float a, float b, floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// First index i in [0, n) with s_indptr[i] >= v (n if none); s_indptr is non-decreasing.
__device__ __forceinline__ int wave_lower_bound(const int *s_indptr, int n, int64_t v) {
    const int lane = threadIdx.x & 63;
    for (int base = 0; base < n; base += 64) {
        const int idx = base + lane;
        const bool pred = idx < n && s_indptr[idx] >= v;
        const unsigned long long m = __ballot(pred);
        if (m) return base + __ffsll(static_cast<long long>(m)) - 1;
    }
    return n;
}

// ------------------------------------------------------------------------------------ units
// A wave walks its stored blocks as a stream of fixed-size "units" of four MFMA steps: 8 blocks
// for 32x1 (2 per v_mfma_f32_32x32x2_f32), 16 for 16x1 (4 per v_mfma_f32_16x16x4_f32, for each
// 16-token half), one block for square shapes.  A unit policy loads a unit's operands into
// registers, issues its MFMAs (all lanes, or only the blocks in an offset range [lo, hi) of the
// unit when it crosses a row end), and stores a finished row tile to Y.

typedef __attribute__((address_space(3))) void lds_void;

// Cache policy of the Y stores: nontemporal (Y is written once and not read here).
constexpr int kStoreNT = 2;

// Destination of one 32-token tile of Y: a buffer resource over the tile's valid rows (rows
// past the last token of the product fall outside it, and the hardware drops those stores).
// The row offset goes in the range-checked vector offset, the column in the scalar offset.
struct TileOut {
    __amdgpu_buffer_rsrc_t rsrc;  // Y + t0 * ldy, over rows * ldy * 4 bytes
    int ldy4;                     // ldy * 4 bytes
};

// Clamp a block column read from memory into [0, Kb) (unsigned compare also catches negatives).
__device__ __forceinline__ int clamp_col(int j, int Kb) {
    return int(min(unsigned(j), unsigned(Kb - 1)));
}

template <int R, int C, bool BF>
struct Unit;

// R x 1 blocks.  For R = 32, lane l supplies block l/32 of a step (A: token l%32 of the X tile;
// B: feature l%32 of the block), acc[v] holds Y[t0 + 8(v/4) + 4(l/32) + v%4][n0 + l%32].
// For R = 16, lane l supplies block l/16 of a step for both token halves, acc.h[h][v] holds
// Y[t0 + 16h + 4(l/16) + v][n0 + l%16].
// With bf16 data the operands are widened to fp32 as they are loaded (exact) and the same fp32
// MFMAs run; the X tile is staged widened to fp32 as well.
template <int R, bool BF>
struct LinearUnit {
    static constexpr int kTokens = 32;      // tokens of the X tile
    static constexpr int kHalves = 1;       // 32-token halves the accumulator spans
    static constexpr int kPer = 64 / R;     // blocks per MFMA step
    static constexpr int kSteps = 4;
    static constexpr int KB = kPer * kSteps;
    static constexpr int kPad = 1;
    static constexpr bool kTileBF16 = false;
    static constexpr bool kTransposed = false;
    struct Ops {
        int j[kSteps];
        float b[kSteps];
    };
    __device__ static int offset_in_step() { return (threadIdx.x & 63) / R; }
    __device__ static int feature() { return (threadIdx.x & 63) % R; }
    // Loads every lane's operands for the unit at p through raw buffer loads over the whole
    // arrays (nnzb blocks): every offset, the unit's included, is in the range-checked vector
    // offset (constant parts go to the instruction's offset field), so lanes past the end of the
    // arrays read 0 and touch no memory.  The descriptors do not depend on p, so a loop over
    // units builds them once.  Lanes past the unit's row segment read the next row's blocks;
    // mask() zeroes them before the MFMAs.
    __device__ static void load(Ops &ops, int p, int nnzb, const int *__restrict__ indices,
                                const void *__restrict__ data) {
        const int o = offset_in_step(), f = feature();
        const __amdgpu_buffer_rsrc_t ri = buffer_rsrc(indices, unsigned(nnzb) * 4u);
        const int vi = (p + o) * 4;
        if constexpr (BF) {
            const __amdgpu_buffer_rsrc_t rd = buffer_rsrc(data, unsigned(nnzb) * (R * 2u));
            const int vd = ((p + o) * R + f) * 2;
#pragma unroll
            for (int m = 0; m < kSteps; ++m) {
                ops.j[m] = __builtin_amdgcn_raw_buffer_load_b32(ri, vi + m * kPer * 4, 0, 0);
                ops.b[m] = __uint_as_float(unsigned(__builtin_amdgcn_raw_buffer_load_b16(
                                               rd, vd + m * kPer * R * 2, 0, 0))
                                           << 16);
            }
        } else {
            const __amdgpu_buffer_rsrc_t rd = buffer_rsrc(data, unsigned(nnzb) * (R * 4u));
            const int vd = ((p + o) * R + f) * 4;
#pragma unroll
            for (int m = 0; m < kSteps; ++m) {
                ops.j[m] = __builtin_amdgcn_raw_buffer_load_b32(ri, vi + m * kPer * 4, 0, 0);
                ops.b[m] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                                         rd, vd + m * kPer * R * 4, 0, 0));
            }
        }
    }
    // Zero the operands of lanes whose block offset in the unit is >= nvalid (partial units).
    __device__ static void mask(Ops &ops, int nvalid) {
        const int o = offset_in_step();
#pragma unroll
        for (int m = 0; m < kSteps; ++m) {
            const bool in = m * kPer + o < nvalid;
            ops.j[m] = in ? ops.j[m] : -1;
            ops.b[m] = in ? ops.b[m] : 0.0f;
        }
    }
};

template <bool BF>
struct Unit<32, 1, BF> : LinearUnit<32, BF> {
    using Ops = typename LinearUnit<32, BF>::Ops;
    using LinearUnit<32, BF>::feature;
    static constexpr int kRegs = 16;
    using Acc = floatx16;
    __device__ static void zero(Acc &acc) {
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[v] = 0.0f;
    }
    // Every element of the tile starts at its column's bias (s_bias: the bias staged in LDS).
    __device__ static void init(Acc &acc, const float *s_bias, int n0) {
        const float b = s_bias[n0 + (threadIdx.x & 31)];
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[v] = b;
    }
    // A unit's X operands, gathered from the LDS tile by gather() and multiplied by mac().
    // Column indices are clamped to [0, Kb]; column Kb of the X tile is the zero pad column
    // that masked lanes point at.
    struct A {
        float a[LinearUnit<32, BF>::kSteps];
    };
    __device__ static void gather(A &x, const Ops &ops, const void *Xs, int XP, int Kb, char *) {
        constexpr int kSteps = LinearUnit<32, BF>::kSteps;
        const float *xrow = static_cast<const float *>(Xs) + feature() * XP;
#pragma unroll
        for (int m = 0; m < kSteps; ++m) x.a[m] = xrow[clamp_col(ops.j[m], Kb + 1)];
    }
    __device__ static void mac(Acc &acc, const A &x, const Ops &ops) {
#pragma unroll
        for (int m = 0; m < LinearUnit<32, BF>::kSteps; ++m) acc = mfma32(x.a[m], ops.b[m], acc);
    }
    __device__ static void mma(Acc &acc, const Ops &ops, const void *Xs, int XP, int Kb,
                               char *wslot) {
        A x;
        gather(x, ops, Xs, XP, Kb, wslot);
        mac(acc, x, ops);
    }
    // Element v of lane l is Y[t0 + 8(v/4) + 4(l/32) + v%4][n0 + l%32].  The row offset of v
    // (uniform) goes in the scalar offset, which the hardware range-checks like the vector
    // offset, so the sixteen stores share one vector offset.
    __device__ static void store(const Acc &acc, const TileOut &o, int n0) {
        const int lane = threadIdx.x & 63, tl = lane & 31, kh = lane >> 5;
        const int vo = 4 * kh * o.ldy4 + tl * 4;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int r = 8 * (v >> 2) + (v & 3);
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc[v]), o.rsrc, vo,
                                                  n0 * 4 + r * o.ldy4, kStoreNT);
        }
    }
    // Register v of every lane alone (v uniform).
    __device__ static void store_reg(float x, const TileOut &o, int n0, int v) {
        const int lane = threadIdx.x & 63, tl = lane & 31, kh = lane >> 5;
        const int r = 8 * (v >> 2) + (v & 3);
        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(x), o.rsrc,
                                              (4 * kh + r) * o.ldy4 + tl * 4, n0 * 4, kStoreNT);
    }
    __device__ static float get(const Acc &acc, int v) { return acc[v]; }
    __device__ static void add(Acc &acc, int v, float x) { acc[v] += x; }
};

template <bool BF>
struct Unit<16, 1, BF> : LinearUnit<16, BF> {
    using Ops = typename LinearUnit<16, BF>::Ops;
    using LinearUnit<16, BF>::feature;
    static constexpr int kRegs = 8;
    struct Acc {
        floatx4 h[2];
    };
    __device__ static void zero(Acc &acc) {
#pragma unroll
        for (int v = 0; v < 4; ++v) acc.h[0][v] = acc.h[1][v] = 0.0f;
    }
    __device__ static void init(Acc &acc, const float *s_bias, int n0) {
        const float b = s_bias[n0 + (threadIdx.x & 15)];
#pragma unroll
        for (int v = 0; v < 4; ++v) acc.h[0][v] = acc.h[1][v] = b;
    }
    struct A {
        float a0[LinearUnit<16, BF>::kSteps], a1[LinearUnit<16, BF>::kSteps];
    };
    __device__ static void gather(A &x, const Ops &ops, const void *Xs, int XP, int Kb, char *) {
        constexpr int kSteps = LinearUnit<16, BF>::kSteps;
        const float *x0 = static_cast<const float *>(Xs) + feature() * XP;
        const float *x1 = x0 + 16 * XP;
#pragma unroll
        for (int m = 0; m < kSteps; ++m) {
            const int j = clamp_col(ops.j[m], Kb + 1);
            x.a0[m] = x0[j];
            x.a1[m] = x1[j];
        }
    }
    __device__ static void mac(Acc &acc, const A &x, const Ops &ops) {
#pragma unroll
        for (int m = 0; m < LinearUnit<16, BF>::kSteps; ++m) {
            acc.h[0] = mfma16(x.a0[m], ops.b[m], acc.h[0]);
            acc.h[1] = mfma16(x.a1[m], ops.b[m], acc.h[1]);
        }
    }
    __device__ static void mma(Acc &acc, const Ops &ops, const void *Xs, int XP, int Kb,
                               char *wslot) {
        A x;
        gather(x, ops, Xs, XP, Kb, wslot);
        mac(acc, x, ops);
    }
    // Element (h, v) of lane l is Y[t0 + 16h + 4(l/16) + v][n0 + l%16].
    __device__ static void store(const Acc &acc, const TileOut &o, int n0) {
        const int lane = threadIdx.x & 63, tl = lane & 15, kq = lane >> 4;
        const int vo = 4 * kq * o.ldy4 + tl * 4;
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int v = 0; v < 4; ++v)
                __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc.h[h][v]), o.rsrc,
                                                      vo + (16 * h + v) * o.ldy4, n0 * 4,
                                                      kStoreNT);
    }
    __device__ static void store_reg(float x, const TileOut &o, int n0, int v) {
        const int lane = threadIdx.x & 63, tl = lane & 15, kq = lane >> 4;
        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(x), o.rsrc,
                                              (4 * kq + 16 * (v >> 2) + (v & 3)) * o.ldy4 + tl * 4,
                                              n0 * 4, kStoreNT);
    }
    __device__ static float get(const Acc &acc, int v) { return acc.h[v >> 2][v & 3]; }
    __device__ static void add(Acc &acc, int v, float x) { acc.h[v >> 2][v & 3] += x; }
};

// LDS transpose read (ds_read_b64_tr_b16): within each group of 16 lanes, lane i receives
// element i % 4 of the 8-byte chunks addressed by lanes 4c + i / 4 of its group, c = 0..3.
__device__ __forceinline__ shortx4 lds_read_tr16(const char *p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_shortx4 *)((__attribute__((address_space(3))) char *)p));
}

// 32x1 bf16 blocks on v_mfma_f32_32x32x16_bf16: the contraction index is the block, 16 blocks
// per instruction, one instruction per unit.  Lane l supplies k-slots 8(l/32) .. +7 for token
// l%32 (A) and feature l%32 (B), i.e. blocks 8(l/32) + e, e = 0..7, of the unit; both operands
// are assembled by transpose reads, four chunks (c = 0..3) per read:
//   * A from the transposed X tile (each column holds the 32 tokens contiguously, 2 bytes each,
//     column pitch XP bf16): lane 4c + q of group g addresses tokens 16(g%2) + 4q .. +3 of
//     column indices[8(g/2) + 4s + c] for read s = 0, 1;
//   * B from a per-wave LDS copy of the unit's blocks ([block][32 features]): the same lane
//     addresses features 16(g%2) + 4q .. +3 of block 8(g/2) + 4s + c.
// Blocks past the segment end read the tile's zero pad column (A) and zero weights (B).
template <>
struct Unit<32, 1, true> {
    static constexpr int kTokens = 32;
    static constexpr int kHalves = 1;
    static constexpr int KB = 16;
    static constexpr int kPad = 0;
    static constexpr bool kTileBF16 = true;
    static constexpr bool kTransposed = true;
    static constexpr int kRegs = 16;
    static constexpr int kSlotBytes = 1024;  // LDS per wave for the unit's blocks
    using Acc = floatx16;
    struct Ops {
        int j[2];   // index for read s
        uintx4 w;   // block l/4, features 8(l%4) .. +7
    };
    __device__ static void zero(Acc &acc) { Unit<32, 1, false>::zero(acc); }
    __device__ static void init(Acc &acc, const float *s_bias, int n0) {
        Unit<32, 1, false>::init(acc, s_bias, n0);
    }
    __device__ static int read_block(int s) {   // block of read s within the unit, this lane
        const int l = threadIdx.x & 63;
        return 8 * (l >> 5) + 4 * s + ((l & 15) >> 2);
    }
    // Offsets in the range-checked vector offset, descriptors over the whole arrays (as for
    // the fp32 linear units).
    __device__ static void load(Ops &ops, int p, int nnzb, const int *__restrict__ indices,
                                const void *__restrict__ data) {
        const int l = threadIdx.x & 63;
        const __amdgpu_buffer_rsrc_t ri = buffer_rsrc(indices, unsigned(nnzb) * 4u);
        const __amdgpu_buffer_rsrc_t rd = buffer_rsrc(data, unsigned(nnzb) * 64u);
        const int io = (p + 8 * (l >> 5) + ((l & 15) >> 2)) * 4;
#pragma unroll
        for (int r = 0; r < 2; ++r)
            ops.j[r] = __builtin_amdgcn_raw_buffer_load_b32(ri, io + 16 * r, 0, 0);
        ops.w = __builtin_amdgcn_raw_buffer_load_b128(rd, p * 64 + l * 16, 0, 0);
    }
    __device__ static void mask(Ops &ops, int nvalid) {
        const int l = threadIdx.x & 63;
#pragma unroll
        for (int r = 0; r < 2; ++r) ops.j[r] = read_block(r) < nvalid ? ops.j[r] : -1;
        ops.w = (l >> 2) < nvalid ? ops.w : uintx4{0u, 0u, 0u, 0u};
    }
    // A from the transposed tile for the two reads of the unit (cols j0, j1 already clamped).
    __device__ static shortx8 gather(const void *Xs, int XP, int j0, int j1) {
        const int l = threadIdx.x & 63, g = l >> 4, q = l & 3;
        const char *xt = static_cast<const char *>(Xs);
        const int tok = (16 * (g & 1) + 4 * q) * 2;   // byte offset within a column
        const shortx4 a0 = lds_read_tr16(xt + j0 * (2 * XP) + tok);
        const shortx4 a1 = lds_read_tr16(xt + j1 * (2 * XP) + tok);
        return __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7);
    }
    // Both operands pass through LDS (A from the tile, B through the wave's block slot), so
    // gather() reads both and mac() only multiplies.
    struct A {
        shortx8 av, bv;
    };
    __device__ static void gather(A &x, const Ops &ops, const void *Xs, int XP, int Kb,
                                  char *wslot) {
        const int l = threadIdx.x & 63, g = l >> 4, c = (l & 15) >> 2, q = l & 3;
        uintx4 *ws = reinterpret_cast<uintx4 *>(wslot);
        ws[l] = ops.w;
        const int tok = (16 * (g & 1) + 4 * q) * 2;
        const int boff = (8 * (g >> 1) + c) * 64 + tok;        // byte offset within the slot
        x.av = gather(Xs, XP, clamp_col(ops.j[0], Kb + 1), clamp_col(ops.j[1], Kb + 1));
        const shortx4 b0 = lds_read_tr16(wslot + boff);
        const shortx4 b1 = lds_read_tr16(wslot + 256 + boff);
        x.bv = __builtin_shufflevector(b0, b1, 0, 1, 2, 3, 4, 5, 6, 7);
    }
    __device__ static void mac(Acc &acc, const A &x, const Ops &) {
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, x.av),
                                                     __builtin_bit_cast(bf16x8, x.bv), acc, 0,
                                                     0, 0);
    }
    __device__ static void mma(Acc &acc, const Ops &ops, const void *Xs, int XP, int Kb,
                               char *wslot) {
        A x;
        gather(x, ops, Xs, XP, Kb, wslot);
        mac(acc, x, ops);
    }
    __device__ static void store(const Acc &acc, const TileOut &o, int n0) {
        Unit<32, 1, false>::store(acc, o, n0);
    }
    __device__ static void store_reg(float x, const TileOut &o, int n0, int v) {
        Unit<32, 1, false>::store_reg(x, o, n0, v);
    }
    __device__ static float get(const Acc &acc, int v) { return acc[v]; }
    __device__ static void add(Acc &acc, int v, float x) { acc[v] += x; }
};

// 32x1 bf16 blocks on 64-token tiles: the unit of Unit<32, 1, true> for two 32-token halves of
// the tile at once.  The halves share the unit's weights (one B operand, loaded once, for two
// v_mfma_f32_32x32x16_bf16), which halves the weight bytes per matrix-core instruction: with
// 32-token tiles the stream of 1 KB weight loads per 32-cycle instruction was bound by the rate
// at which a CU's texture addresser takes vector loads (its busy counter near saturation during
// the stream, on MI355X).  The transposed tile holds the halves one after the other, each laid
// out as Unit<32, 1, true>'s tile (K + 1 columns of 32 tokens, column pitch 72 bytes); each
// half's sums are those of the 32-token unit over the same blocks.
struct Unit64BF {
    using Half = Unit<32, 1, true>;
    static constexpr int KB = 16;
    static constexpr int kPad = 0;
    static constexpr bool kTileBF16 = true;
    static constexpr bool kTransposed = true;
    static constexpr int kTokens = 64;
    static constexpr int kHalves = 2;
    static constexpr int kRegs = 32;
    using Ops = Half::Ops;
    struct Acc {
        floatx16 a[2];
    };
    // Bytes from a column of the first half of the tile to the same column of the second.
    __device__ static int half_bytes(int Kb) { return (Kb + 1) * 72; }
    __device__ static void zero(Acc &acc) {
        Half::zero(acc.a[0]);
        Half::zero(acc.a[1]);
    }
    __device__ static void init(Acc &acc, const float *s_bias, int n0) {
        Half::init(acc.a[0], s_bias, n0);
        Half::init(acc.a[1], s_bias, n0);
    }
    __device__ static void load(Ops &ops, int p, int nnzb, const int *__restrict__ indices,
                                const void *__restrict__ data) {
        Half::load(ops, p, nnzb, indices, data);
    }
    __device__ static void mask(Ops &ops, int nvalid) { Half::mask(ops, nvalid); }
    struct A {
        shortx8 av[2], bv;
    };
    __device__ static void gather(A &x, const Ops &ops, const void *Xs, int XP, int Kb,
                                  char *wslot) {
        const int l = threadIdx.x & 63, g = l >> 4, c = (l & 15) >> 2, q = l & 3;
        uintx4 *ws = reinterpret_cast<uintx4 *>(wslot);
        ws[l] = ops.w;
        const int tok = (16 * (g & 1) + 4 * q) * 2;
        const int boff = (8 * (g >> 1) + c) * 64 + tok;
        const int j0 = clamp_col(ops.j[0], Kb + 1), j1 = clamp_col(ops.j[1], Kb + 1);
        x.av[0] = Half::gather(Xs, XP, j0, j1);
        x.av[1] = Half::gather(static_cast<const char *>(Xs) + half_bytes(Kb), XP, j0, j1);
        const shortx4 b0 = lds_read_tr16(wslot + boff);
        const shortx4 b1 = lds_read_tr16(wslot + 256 + boff);
        x.bv = __builtin_shufflevector(b0, b1, 0, 1, 2, 3, 4, 5, 6, 7);
    }
    __device__ static void mac(Acc &acc, const A &x, const Ops &) {
#pragma unroll
        for (int h = 0; h < 2; ++h)
            acc.a[h] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                __builtin_bit_cast(bf16x8, x.av[h]), __builtin_bit_cast(bf16x8, x.bv), acc.a[h],
                0, 0, 0);
    }
    // Half h of the tile: its 32 tokens start 32 h rows into the tile's Y window.
    __device__ static void store_half(const Acc &acc, const TileOut &o, int n0, int h) {
        const int lane = threadIdx.x & 63, tl = lane & 31, kh = lane >> 5;
        const int vo = 4 * kh * o.ldy4 + tl * 4;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int r = 32 * h + 8 * (v >> 2) + (v & 3);
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc.a[h][v]), o.rsrc, vo,
                                                  n0 * 4 + r * o.ldy4, kStoreNT);
        }
    }
    __device__ static void store(const Acc &acc, const TileOut &o, int n0) {
        store_half(acc, o, n0, 0);
        store_half(acc, o, n0, 1);
    }
    // Register v (uniform, 0 .. 31): half v / 16, register v % 16 of the 32-token layout.
    __device__ static void store_reg(float x, const TileOut &o, int n0, int v) {
        const int lane = threadIdx.x & 63, tl = lane & 31, kh = lane >> 5, vv = v & 15;
        const int r = 32 * (v >> 4) + 8 * (vv >> 2) + (vv & 3);
        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(x), o.rsrc,
                                              (4 * kh + r) * o.ldy4 + tl * 4, n0 * 4, kStoreNT);
    }
    __device__ static float get(const Acc &acc, int v) { return acc.a[v >> 4][v & 15]; }
    __device__ static void add(Acc &acc, int v, float x) { acc.a[v >> 4][v & 15] += x; }
};

// ------------------------------------------------------------------------- planned units
// A plan (prepared once per matrix) stores, for every unit of KB blocks of one block-row (the
// last unit of a row padded with zero blocks whose column is the tile's zero pad column), its
// block columns and its weights already in the lane order of the unit's MFMAs, so that a
// unit's operands arrive in two 16-byte loads per lane (one for the columns, one for the
// weights) and no operand is masked or re-arranged at run time.  The sums are those of the
// unplanned unit of the same shape: the same blocks in the same k-slots of the same
// instructions.  Loads of a unit at or past `ulim` fetch nothing and return 0 (the unit's
// offset is in the range-checked vector offset).
template <int R, int C, bool BF>
struct PlanUnit;

// fp32 32x1: unit = 8 blocks, four v_mfma_f32_32x32x2_f32 steps; step m of half h = l/32 takes
// block 2m + h.  Columns: cols[u][h][m] as byte offsets into a row of the X tile, 4 * col with
// col clamped to [0, Kb] (Kb: the tile's zero pad column), so a gather is one add (32 bytes per
// unit); weights: vals[u][l][m] = block (2m + l/32), feature l%32 (1 KB per unit).  The unit's
// offset goes in the scalar offset of the loads (range-checked like the vector offset), so a
// unit's loads need no per-lane arithmetic.
template <>
struct PlanUnit<32, 1, false> {
    using Base = Unit<32, 1, false>;
    static constexpr int KB = 8;
    static constexpr int kColBytes = 32;
    static constexpr int kValBytes = 1024;
    static constexpr int kColScale = 4;   // bytes per column in a row of the X tile
    struct Ops {
        uintx4 j;
        floatx4 b;
    };
    __device__ static void load(Ops &ops, int u, int ulim, const int32_t *__restrict__ cols,
                                const void *__restrict__ vals) {
        const int l = threadIdx.x & 63;
        const __amdgpu_buffer_rsrc_t rc = buffer_rsrc(cols, unsigned(ulim) * kColBytes);
        const __amdgpu_buffer_rsrc_t rv = buffer_rsrc(vals, unsigned(ulim) * kValBytes);
        ops.j = __builtin_amdgcn_raw_buffer_load_b128(rc, (l >> 5) * 16, u * kColBytes, 0);
        ops.b = __builtin_bit_cast(
            floatx4, __builtin_amdgcn_raw_buffer_load_b128(rv, l * 16, u * kValBytes, 0));
    }
    using A = typename Base::A;
    __device__ static void gather(A &x, const Ops &ops, const void *Xs, int XP, int, char *) {
        const char *xrow = static_cast<const char *>(Xs) + (threadIdx.x & 31) * XP * 4;
#pragma unroll
        for (int m = 0; m < 4; ++m) x.a[m] = *reinterpret_cast<const float *>(xrow + ops.j[m]);
    }
    __device__ static void mac(typename Base::Acc &acc, const A &x, const Ops &ops) {
#pragma unroll
        for (int m = 0; m < 4; ++m) acc = mfma32(x.a[m], ops.b[m], acc);
    }
};

// bf16 32x1: unit = 16 blocks, one v_mfma_f32_32x32x16_bf16.  Columns: cols[u][h][c][s] =
// block 8h + 4s + c as byte offsets of its column in the transposed X tile (column pitch 72
// bytes: kColScale * col, col clamped to [0, Kb]); lane l reads the pair of (h, c) = (l/32,
// (l%16)/4) (64 bytes per unit).  Weights: vals[u][l][e] = block 8(l/32) + e, feature l%32, as
// bf16 (16 bytes per lane, 1 KB per unit) -- exactly the B operand, so no LDS round trip.
template <>
struct PlanUnit<32, 1, true> {
    using Base = Unit<32, 1, true>;
    static constexpr int KB = 16;
    static constexpr int kColBytes = 64;
    static constexpr int kValBytes = 1024;
    static constexpr int kColScale = 72;  // bytes per column of the transposed tile (pitch 36)
    struct Ops {
        uintx2 j;
        uintx4 b;
    };
    __device__ static void load(Ops &ops, int u, int ulim, const int32_t *__restrict__ cols,
                                const void *__restrict__ vals) {
        const int l = threadIdx.x & 63;
        const __amdgpu_buffer_rsrc_t rc = buffer_rsrc(cols, unsigned(ulim) * kColBytes);
        const __amdgpu_buffer_rsrc_t rv = buffer_rsrc(vals, unsigned(ulim) * kValBytes);
        ops.j = __builtin_amdgcn_raw_buffer_load_b64(rc, ((l >> 5) * 4 + ((l & 15) >> 2)) * 8,
                                                     u * kColBytes, 0);
        ops.b = __builtin_amdgcn_raw_buffer_load_b128(rv, l * 16, u * kValBytes, 0);
    }
    struct A {
        shortx8 av;
    };
    __device__ static void gather(A &x, const Ops &ops, const void *Xs, int, int, char *) {
        const int l = threadIdx.x & 63, g = l >> 4, q = l & 3;
        const char *xt = static_cast<const char *>(Xs) + (16 * (g & 1) + 4 * q) * 2;
        const shortx4 a0 = lds_read_tr16(xt + ops.j[0]);
        const shortx4 a1 = lds_read_tr16(xt + ops.j[1]);
        x.av = __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7);
    }
    __device__ static void mac(typename Base::Acc &acc, const A &x, const Ops &ops) {
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, x.av),
                                                     __builtin_bit_cast(bf16x8, ops.b), acc, 0,
                                                     0, 0);
    }
};

// 32x1 blocks on the bf16 matrix cores with the X operand gathered from the row-major fp32 X
// tile (32 tokens of one column per half-wave: one conflict-free ds_read_b32 per block) and
// the weights from a plan holding NP bf16 pieces of every weight, each piece an operand plane
// in MFMA lane order.  NP = 3: fp32 data, a plan of arithmetic BSR_ARITH_BF16X3.  A finite
// fp32 value v is the sum v0 + v1 + v2 of three bf16 values: v0 = v with its low 16 bits
// cleared, r = v - v0 (exact), v1 = r with its low 16 bits cleared, v2 = r - v1 (exact, at most
// 8 significant bits), so |v1| < 2^-7 |v| and |v2| < 2^-14 |v|.  Of the nine cross terms of
// x * w the six with i + j <= 2 are formed (each product of two bf16 values is exact in fp32)
// and the three left out sum to less than 2^-20 |x w|.  The six v_mfma_f32_32x32x16_bf16 run
// smallest first into the one fp32 accumulator.
// Unit = 16 blocks; lane l supplies k-slots 8(l/32) .. +7, i.e. blocks 8(l/32) + e, for token
// l%32 (A: gathered, then split in registers) and feature l%32 (B).
// Columns: cols[u][h][e] = 4 * column of block 8h + e as uint16 byte offsets into a row of the
// fp32 tile (column clamped to [0, Kb]; 32 bytes per unit, one 16-byte load per lane).
// Weights: vals[u][p][l][e] = piece p of block 8(l/32) + e, feature l%32 (NP planes of 1 KB
// per unit, each exactly a B operand).
template <int NP>
struct GatherPlanUnit {
    static_assert(NP == 3, "three pieces per fp32 weight");
    using Base = Unit<32, 1, false>;
    static constexpr int KB = 16;
    static constexpr int kColBytes = 32;
    static constexpr int kPlaneBytes = 1024;
    static constexpr int kValBytes = NP * kPlaneBytes;
    static constexpr int kColScale = 4;   // bytes per column in a row of the X tile
    static constexpr int kMaxColBytes = 65535;
    struct Ops {
        uintx4 j;       // byte offsets of blocks 8(l/32) + e, two per word (e even: low half)
        uintx4 b[NP];   // the weight pieces, bf16 pairs
    };
    __device__ static void load(Ops &ops, int u, int ulim, const int32_t *__restrict__ cols,
                                const void *__restrict__ vals) {
        const int l = threadIdx.x & 63;
        const __amdgpu_buffer_rsrc_t rc = buffer_rsrc(cols, unsigned(ulim) * kColBytes);
        const __amdgpu_buffer_rsrc_t rv = buffer_rsrc(vals, unsigned(ulim) * kValBytes);
        ops.j = __builtin_amdgcn_raw_buffer_load_b128(rc, (l >> 5) * 16, u * kColBytes, 0);
#pragma unroll
        for (int p = 0; p < NP; ++p)
            ops.b[p] = __builtin_amdgcn_raw_buffer_load_b128(rv, p * kPlaneBytes + l * 16,
                                                             u * kValBytes, 0);
    }
    // The bf16 upper halves of two fp32 words, as one packed pair (a low, b high).
    __device__ static unsigned hi_pair(unsigned a, unsigned b) {
        return __builtin_amdgcn_perm(b, a, 0x07060302u);
    }
    // The gathered fp32 values; the split happens in mac().
    struct A {
        float v[8];
    };
    __device__ static void gather(A &x, const Ops &ops, const void *Xs, int XP, int, char *) {
        const char *xrow = static_cast<const char *>(Xs) + (threadIdx.x & 31) * XP * 4;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const unsigned w = ops.j[e >> 1];
            const unsigned off = (e & 1) ? (w >> 16) : (w & 0xffffu);
            x.v[e] = *reinterpret_cast<const float *>(xrow + off);
        }
    }
    __device__ static void mac(typename Base::Acc &acc, const A &x, const Ops &ops) {
        uintx4 x0, x1, x2;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            unsigned r[2], c[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const float a = x.v[2 * q + i];
                const float rr = a - __uint_as_float(__float_as_uint(a) & 0xffff0000u);
                const float cc = rr - __uint_as_float(__float_as_uint(rr) & 0xffff0000u);
                r[i] = __float_as_uint(rr);
                c[i] = __float_as_uint(cc);
            }
            x0[q] = hi_pair(__float_as_uint(x.v[2 * q]), __float_as_uint(x.v[2 * q + 1]));
            x1[q] = hi_pair(r[0], r[1]);
            x2[q] = hi_pair(c[0], c[1]);
        }
        auto mf = [&](const uintx4 &a, const uintx4 &b) {
            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                         __builtin_bit_cast(bf16x8, b), acc, 0,
                                                         0, 0);
        };
        mf(x2, ops.b[0]);
        mf(x1, ops.b[1]);
        mf(x0, ops.b[2]);
        mf(x1, ops.b[0]);
        mf(x0, ops.b[1]);
        mf(x0, ops.b[0]);
    }
};
using SplitPlanUnit = GatherPlanUnit<3>;

// Planned 32x1 bf16 blocks on 64-token tiles: PlanUnit<32, 1, true>'s operands (the same plan)
// multiplied into both halves of Unit64BF's tile.
struct PlanUnit64BF {
    using Base = Unit64BF;
    using One = PlanUnit<32, 1, true>;
    static constexpr int KB = One::KB;
    static constexpr int kColBytes = One::kColBytes;
    static constexpr int kValBytes = One::kValBytes;
    static constexpr int kColScale = One::kColScale;
    using Ops = One::Ops;
    __device__ static void load(Ops &ops, int u, int ulim, const int32_t *__restrict__ cols,
                                const void *__restrict__ vals) {
        One::load(ops, u, ulim, cols, vals);
    }
    struct A {
        shortx8 av[2];
    };
    __device__ static void gather(A &x, const Ops &ops, const void *Xs, int XP, int Kb,
                                  char *wslot) {
        typename One::A h0, h1;
        One::gather(h0, ops, Xs, XP, Kb, wslot);
        One::gather(h1, ops, static_cast<const char *>(Xs) + Unit64BF::half_bytes(Kb), XP, Kb,
                    wslot);
        x.av[0] = h0.av;
        x.av[1] = h1.av;
    }
    __device__ static void mac(Unit64BF::Acc &acc, const A &x, const Ops &ops) {
#pragma unroll
        for (int h = 0; h < 2; ++h)
            acc.a[h] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                __builtin_bit_cast(bf16x8, x.av[h]), __builtin_bit_cast(bf16x8, ops.b), acc.a[h],
                0, 0, 0);
    }
};

// Accumulator, bias and store plumbing shared by the square units (the output layouts of the
// 32x32 and 16x16 MFMAs do not depend on the input type).
template <int R>
using LinearBase = Unit<R, 1, false>;

// 32x32 fp32 blocks, v_mfma_f32_32x32x2_f32.  Lane l loads columns 8u + 4(l/32) .. +3 of block
// row l%32 (u = 0..3); for step (u, e) its k-slot l/32 stands for c = 8u + 4(l/32) + e in both
// operands.
template <>
struct Unit<32, 32, false> {
    static constexpr int KB = 1;
    static constexpr int kPad = 4;
    static constexpr bool kTileBF16 = false;
    static constexpr bool kTransposed = false;
    static constexpr int kRegs = 16;
    using Acc = floatx16;
    struct Ops {
        int j;
        floatx4 d[4];
    };
    __device__ static void zero(Acc &acc) { LinearBase<32>::zero(acc); }
    __device__ static void init(Acc &acc, const float *s_bias, int n0) {
        LinearBase<32>::init(acc, s_bias, n0);
    }
    __device__ static void mask(Ops &, int) {}
    // Range-checked loads based at the unit, as for the R x 1 units: a position at or past
    // nnzb reads 0 and touches no memory.
    __device__ static void load(Ops &ops, int p, int nnzb, const int *__restrict__ indices,
                                const void *__restrict__ data) {
        const int lane = threadIdx.x & 63, tl = lane & 31, kh = lane >> 5;
        const __amdgpu_buffer_rsrc_t ri = buffer_rsrc(indices, unsigned(nnzb) * 4u);
        const __amdgpu_buffer_rsrc_t rd = buffer_rsrc(data, unsigned(nnzb) * 4096u);
        ops.j = uniform(__builtin_amdgcn_raw_buffer_load_b32(ri, p * 4, 0, 0));
        const int vd = p * 4096 + (tl * 8 + kh) * 16;
#pragma unroll
        for (int u = 0; u < 4; ++u)
            ops.d[u] = __builtin_bit_cast(
                floatx4, __builtin_amdgcn_raw_buffer_load_b128(rd, vd + 32 * u, 0, 0));
    }
    __device__ static void mma(Acc &acc, const Ops &ops, const void *Xs, int XP, int Kb,
                                    char *) {
        const int lane = threadIdx.x & 63, tl = lane & 31, kh = lane >> 5;
        const float *xb =
            static_cast<const float *>(Xs) + tl * XP + 4 * kh + clamp_col(ops.j, Kb) * 32;
        floatx4 a[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) a[u] = *reinterpret_cast<const floatx4 *>(xb + 8 * u);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
#pragma unroll
            for (int e = 0; e < 4; ++e) acc = mfma32(a[u][e], ops.d[u][e], acc);
        }
    }
    __device__ static void store(const Acc &acc, const TileOut &o, int n0) {
        LinearBase<32>::store(acc, o, n0);
    }
    __device__ static void store_reg(float x, const TileOut &o, int n0, int v) {
        LinearBase<32>::store_reg(x, o, n0, v);
    }
    __device__ static float get(const Acc &acc, int v) { return acc[v]; }
    __device__ static void add(Acc &acc, int v, float x) { acc[v] += x; }
};

// 32x32 bf16 blocks, v_mfma_f32_32x32x16_bf16, two instructions per block.  For half u of the
// block's columns, lane l supplies k-slots 8(l/32) .. +7, standing for c = 16u + 8(l/32) + e:
// 16 contiguous bytes of token l%32's X row (from the bf16 LDS tile) and of block row l%32.
template <>
struct Unit<32, 32, true> {
    static constexpr int KB = 1;
    static constexpr int kPad = 8;
    static constexpr bool kTileBF16 = true;
    static constexpr bool kTransposed = false;
    static constexpr int kRegs = 16;
    using Acc = floatx16;
    struct Ops {
        int j;
        uintx4 d[2];
    };
    __device__ static void zero(Acc &acc) { LinearBase<32>::zero(acc); }
    __device__ static void init(Acc &acc, const float *s_bias, int n0) {
        LinearBase<32>::init(acc, s_bias, n0);
    }
    __device__ static void mask(Ops &, int) {}
    __device__ static void load(Ops &ops, int p, int nnzb, const int *__restrict__ indices,
                                const void *__restrict__ data) {
        const int lane = threadIdx.x & 63, tl = lane & 31, kh = lane >> 5;
        const __amdgpu_buffer_rsrc_t ri = buffer_rsrc(indices, unsigned(nnzb) * 4u);
        const __amdgpu_buffer_rsrc_t rd = buffer_rsrc(data, unsigned(nnzb) * 2048u);
        ops.j = uniform(__builtin_amdgcn_raw_buffer_load_b32(ri, p * 4, 0, 0));
        const int vd = p * 2048 + (tl * 4 + kh) * 16;
#pragma unroll
        for (int u = 0; u < 2; ++u)
            ops.d[u] = __builtin_amdgcn_raw_buffer_load_b128(rd, vd + 32 * u, 0, 0);
    }
    __device__ static void mma(Acc &acc, const Ops &ops, const void *Xs, int XP, int Kb,
                                    char *) {
        const int lane = threadIdx.x & 63, tl = lane & 31, kh = lane >> 5;
        const bf16_t *xb =
            static_cast<const bf16_t *>(Xs) + tl * XP + 8 * kh + clamp_col(ops.j, Kb) * 32;
        uintx4 a[2];
#pragma unroll
        for (int u = 0; u < 2; ++u) a[u] = *reinterpret_cast<const uintx4 *>(xb + 16 * u);
#pragma unroll
        for (int u = 0; u < 2; ++u)
            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a[u]),
                                                         __builtin_bit_cast(bf16x8, ops.d[u]),
                                                         acc, 0, 0, 0);
    }
    __device__ static void store(const Acc &acc, const TileOut &o, int n0) {
        LinearBase<32>::store(acc, o, n0);
    }
    __device__ static void store_reg(float x, const TileOut &o, int n0, int v) {
        LinearBase<32>::store_reg(x, o, n0, v);
    }
    __device__ static float get(const Acc &acc, int v) { return acc[v]; }
    __device__ static void add(Acc &acc, int v, float x) { acc[v] += x; }
};

// 16x16 fp32 blocks, v_mfma_f32_16x16x4_f32 on two 16-token halves.  Lane l loads row l%16,
// columns 4(l/16)..+3 of the block (the whole block in one instruction); k-slot l/16 of step e
// stands for c = 4(l/16) + e.
// 16x16 blocks, KBN blocks per unit (1, or 4 for rows with many blocks: one memory round trip
// then feeds eight MFMAs instead of two).  A partial unit skips its missing blocks (their index
// is set to -1), so no zero weight meets an infinite X element.
//   fp32: v_mfma_f32_16x16x4_f32 on two 16-token halves.  Lane l loads row l%16, columns
//   4(l/16)..+3 of the block (the whole block in one instruction); k-slot l/16 of step e stands
//   for c = 4(l/16) + e.
//   bf16: v_mfma_f32_16x16x16_bf16 on two 16-token halves, one instruction per block and half.
//   Lane l supplies k-slots 4(l/16) .. +3, standing for c = 4(l/16) + e: 8 contiguous bytes of
//   token l%16's X row and of block row l%16.
template <bool BF, int KBN>
struct Unit1616 {
    static constexpr int KB = KBN;
    static constexpr int kPad = 8;
    static constexpr bool kTileBF16 = BF;
    static constexpr bool kTransposed = false;
    static constexpr int kRegs = 8;
    static constexpr int kBlockBytes = BF ? 512 : 1024;
    using Acc = typename LinearBase<16>::Acc;
    using Data = typename std::conditional<BF, uintx2, floatx4>::type;
    struct Ops {
        int j[KB];
        Data d[KB];
    };
    __device__ static void zero(Acc &acc) { LinearBase<16>::zero(acc); }
    __device__ static void init(Acc &acc, const float *s_bias, int n0) {
        LinearBase<16>::init(acc, s_bias, n0);
    }
    __device__ static void mask(Ops &ops, int nvalid) {
#pragma unroll
        for (int u = 1; u < KB; ++u) ops.j[u] = u < nvalid ? ops.j[u] : -1;
    }
    __device__ static void load(Ops &ops, int p, int nnzb, const int *__restrict__ indices,
                                const void *__restrict__ data) {
        const int lane = threadIdx.x & 63;
        const __amdgpu_buffer_rsrc_t ri = buffer_rsrc(indices, unsigned(nnzb) * 4u);
        const __amdgpu_buffer_rsrc_t rd = buffer_rsrc(data, unsigned(nnzb) * unsigned(kBlockBytes));
        if constexpr (KB == 1) {
            ops.j[0] = uniform(__builtin_amdgcn_raw_buffer_load_b32(ri, p * 4, 0, 0));
        } else {
            static_assert(KB == 4, "one 16-byte load of the unit's indices");
            const uintx4 jj = __builtin_amdgcn_raw_buffer_load_b128(ri, p * 4, 0, 0);
#pragma unroll
            for (int u = 0; u < KB; ++u) ops.j[u] = uniform(int(jj[u]));
        }
        const int off = p * kBlockBytes + ((lane & 15) * 4 + (lane >> 4)) * (BF ? 8 : 16);
#pragma unroll
        for (int u = 0; u < KB; ++u) {
            if constexpr (BF)
                ops.d[u] = __builtin_amdgcn_raw_buffer_load_b64(rd, off + kBlockBytes * u, 0, 0);
            else
                ops.d[u] = __builtin_bit_cast(
                    floatx4, __builtin_amdgcn_raw_buffer_load_b128(rd, off + kBlockBytes * u, 0, 0));
        }
    }
    __device__ static void mma(Acc &acc, const Ops &ops, const void *Xs, int XP, int Kb,
                                    char *) {
        const int lane = threadIdx.x & 63, tl = lane & 15, kq = lane >> 4;
#pragma unroll
        for (int u = 0; u < KB; ++u) {
            if (u > 0 && ops.j[u] < 0) break;   // the rest of a partial unit
            const int col = clamp_col(ops.j[u], Kb) * 16;
            if constexpr (BF) {
                const bf16_t *xb = static_cast<const bf16_t *>(Xs) + tl * XP + 4 * kq + col;
                const uintx2 a0 = *reinterpret_cast<const uintx2 *>(xb);
                const uintx2 a1 = *reinterpret_cast<const uintx2 *>(xb + 16 * XP);
                const shortx4 b = __builtin_bit_cast(shortx4, ops.d[u]);
                acc.h[0] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(
                    __builtin_bit_cast(shortx4, a0), b, acc.h[0], 0, 0, 0);
                acc.h[1] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(
                    __builtin_bit_cast(shortx4, a1), b, acc.h[1], 0, 0, 0);
            } else {
                const float *xb = static_cast<const float *>(Xs) + tl * XP + 4 * kq + col;
                const floatx4 a0 = *reinterpret_cast<const floatx4 *>(xb);
                const floatx4 a1 = *reinterpret_cast<const floatx4 *>(xb + 16 * XP);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    acc.h[0] = mfma16(a0[e], ops.d[u][e], acc.h[0]);
                    acc.h[1] = mfma16(a1[e], ops.d[u][e], acc.h[1]);
                }
            }
        }
    }
    __device__ static void store(const Acc &acc, const TileOut &o, int n0) {
        LinearBase<16>::store(acc, o, n0);
    }
    __device__ static void store_reg(float x, const TileOut &o, int n0, int v) {
        LinearBase<16>::store_reg(x, o, n0, v);
    }
    __device__ static float get(const Acc &acc, int v) { return LinearBase<16>::get(acc, v); }
    __device__ static void add(Acc &acc, int v, float x) { LinearBase<16>::add(acc, v, x); }
};

template <>
struct Unit<16, 16, false> : Unit1616<false, 1> {};
template <>
struct Unit<16, 16, true> : Unit1616<true, 1> {};

// The unit a kernel instantiation runs: Unit<R, C, BF>, or (W = 4) the four-block 16x16 unit.
template <int R, int C, bool BF, int W>
struct UnitOf {
    using type = Unit<R, C, BF>;
};
template <bool BF>
struct UnitOf<16, 16, BF, 4> {
    using type = Unit1616<BF, 4>;
};

}  // namespace

}  // namespace bsr
