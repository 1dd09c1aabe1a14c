// LDS-tiled BSR product on the vector ALUs, for block shapes without a matrix-core kernel:
// one-row blocks 1 x C (1x1 .. 1x32), narrow column blocks 2x1 .. 8x1 and small squares 2x2,
// 4x4, 8x8; fp32 or bf16 inputs, fp32 accumulation, fp32 output.
//
// Y[t][n] = bias[n] + sum over stored blocks p of block-row i = n / R of
//           sum over c < C of X[t][indices[p] * C + c] * data[p][n - iR][c]          (Sec. 2.2)
//
// For R = 1 the rows of W share no input columns, so the product has no dense contraction to
// hand to the matrix cores; for 2x1 .. 8x8 a matrix-core tile would be mostly padding.  These
// shapes run as fp32 fused multiply-adds:
//   * one workgroup = a 32-token tile x a slice of block-rows (equal row counts); the X tile
//     [32][K] is staged once into LDS as fp32 (bf16 widened, exactly) with a row pitch XP that
//     makes a read of one column segment by the 32 tokens hit distinct banks;
//   * each wave walks whole block-rows of the slice, round robin; lane l is token l % 32 of
//     half l / 32, and the two halves take alternate chunks of U blocks of the row;
//   * a lane accumulates the R outputs of its token over its chunks in fp32 (block column c
//     outer, output row r inner); the halves are summed at the row end (both halves then hold
//     the same bits) and each half stores its share of Y[t][iR .. iR + R);
//   * the weights of a chunk are read from global memory by all 32 lanes of a half (a
//     broadcast), double-buffered in registers one chunk ahead; X comes from LDS.
// The summation order depends only on the launch shape, so results are bitwise reproducible.
#include <type_traits>
#include <utility>

#include "device_common.h"
#include "spmm_tiled.h"

namespace bsr {

namespace {

typedef float floatx2 __attribute__((ext_vector_type(2)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef unsigned uintx2 __attribute__((ext_vector_type(2)));
typedef unsigned uintx4 __attribute__((ext_vector_type(4)));

constexpr int kVT = 32;   // tokens per workgroup

template <int R, int C>
struct VShape {
    static constexpr int RC = R * C;
    // Blocks per chunk: about 32 weights per chunk, at most 8 blocks.
    static constexpr int U = RC >= 32 ? 1 : (32 / RC > 8 ? 8 : 32 / RC);
    static constexpr int NWORDS = U * RC;   // weights per chunk
    // Width of the LDS reads of a block's X segment (C is a multiple of it).
    static constexpr int VW = C % 4 == 0 ? 4 : (C % 2 == 0 ? 2 : 1);
    // Waves per workgroup: 16 (128 registers per lane) for chunks of up to 16 weights, else 8
    // (256 registers: two chunks in flight plus the X segments they read).
    static constexpr int NW = NWORDS <= 16 ? 16 : 8;
    static_assert(NWORDS % 8 == 0, "a chunk's weights are whole 16-byte loads of bf16 or fp32");
};

template <int N>
struct VecOf;
template <>
struct VecOf<1> {
    typedef float type;
};
template <>
struct VecOf<2> {
    typedef floatx2 type;
};
template <>
struct VecOf<4> {
    typedef floatx4 type;
};

// Operands of one chunk: U block columns and U * R * C weights (fp32).
// Waves per workgroup: per-lane weights (bf16) need registers for two chunks, so wide chunks
// get 8 waves (VShape::NW); broadcast weights (fp32) take at most four registers a chunk, so
// every shape gets 16.
template <int R, int C, bool BF>
constexpr int kWaves = BF ? VShape<R, C>::NW : 16;

template <int R, int C>
struct VOps {
    int j[VShape<R, C>::U];
    float w[VShape<R, C>::NWORDS];
};

// Loads the chunk that starts `o` blocks into the row (the row's arrays are the buffer ranges
// ri / rd and every offset is in the range-checked vector offset, so a chunk past the row end
// reads 0 and touches no memory).
template <int R, int C, bool BF>
__device__ __forceinline__ void vload(VOps<R, C> &ops, __amdgpu_buffer_rsrc_t ri,
                                      __amdgpu_buffer_rsrc_t rd, int o) {
    using S = VShape<R, C>;
    if constexpr (S::U == 8) {
        const uintx4 a = __builtin_amdgcn_raw_buffer_load_b128(ri, o * 4, 0, 0);
        const uintx4 b = __builtin_amdgcn_raw_buffer_load_b128(ri, o * 4 + 16, 0, 0);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            ops.j[u] = int(a[u]);
            ops.j[4 + u] = int(b[u]);
        }
    } else if constexpr (S::U == 4) {
        const uintx4 a = __builtin_amdgcn_raw_buffer_load_b128(ri, o * 4, 0, 0);
#pragma unroll
        for (int u = 0; u < 4; ++u) ops.j[u] = int(a[u]);
    } else if constexpr (S::U == 2) {
        const uintx2 a = __builtin_amdgcn_raw_buffer_load_b64(ri, o * 4, 0, 0);
        ops.j[0] = int(a[0]);
        ops.j[1] = int(a[1]);
    } else {
        ops.j[0] = int(__builtin_amdgcn_raw_buffer_load_b32(ri, o * 4, 0, 0));
    }
    if constexpr (BF) {
        // 8 bf16 weights per 16-byte load, widened exactly to fp32.
#pragma unroll
        for (int q = 0; q < S::NWORDS / 8; ++q) {
            const uintx4 v = __builtin_amdgcn_raw_buffer_load_b128(rd, o * (S::RC * 2) + 16 * q, 0, 0);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                ops.w[8 * q + 2 * e] = __uint_as_float(v[e] << 16);
                ops.w[8 * q + 2 * e + 1] = __uint_as_float(v[e] & 0xffff0000u);
            }
        }
    } else {
#pragma unroll
        for (int q = 0; q < S::NWORDS / 4; ++q) {
            const uintx4 v = __builtin_amdgcn_raw_buffer_load_b128(rd, o * (S::RC * 4) + 16 * q, 0, 0);
#pragma unroll
            for (int e = 0; e < 4; ++e) ops.w[4 * q + e] = __uint_as_float(v[e]);
        }
    }
}

// acc[r] += sum over the chunk's first nv blocks (all U when !MASKED) and their columns c of
// X[t][j * C + c] * w[r][c].  xrow is this lane's token row of the LDS tile.  Block columns are
// clamped into [0, Kb), so a malformed index reads a wrong column of the tile, never outside it.
// jlo: the tile's first block column (0 for a whole-row tile; the chunk's first column for the
// column-chunked kernel); columns are clamped into [jlo, jlo + Kb).
template <int R, int C, bool MASKED>
__device__ __forceinline__ void vcompute(float (&acc)[R], const VOps<R, C> &ops,
                                         const float *xrow, int Kb, int nv, int jlo = 0) {
    using S = VShape<R, C>;
    using V = typename VecOf<S::VW>::type;
#pragma unroll
    for (int u = 0; u < S::U; ++u) {
        if (MASKED && u >= nv) break;
        const unsigned col = min(unsigned(ops.j[u] - jlo), unsigned(Kb - 1)) * unsigned(C);
        const float *xs = xrow + col;
#pragma unroll
        for (int c0 = 0; c0 < C; c0 += S::VW) {
            const V xv = *reinterpret_cast<const V *>(xs + c0);
#pragma unroll
            for (int cc = 0; cc < S::VW; ++cc) {
                float x;
                if constexpr (S::VW == 1) x = xv;
                else x = xv[cc];
#pragma unroll
                for (int r = 0; r < R; ++r)
                    acc[r] = __builtin_fmaf(x, ops.w[u * S::RC + r * C + c0 + cc], acc[r]);
            }
        }
    }
}

// fp32 weights through lane broadcasts.  Loading every weight of a chunk into every lane (the
// loads above) made these kernels bound by the rate at which a CU's texture addresser takes
// vector loads (about 0.8 of its cycles busy on the 4096-token FFN rows, the vector ALUs under
// 0.25, MI355X counters).  Instead, each 16-lane row of a half holds 16 words of its half's
// chunk, one word per lane (both rows of a half the same words), so a chunk of NWORDS weights
// costs ceil(NWORDS / 16) dword loads, and every multiply-add reads its weight with a DPP row
// broadcast (v_fmac_f32 with row_newbcast: each row gets the value of one of its lanes).  The
// chunk's block columns arrive the same way, one per lane, and are broadcast before use.
template <int R, int C>
struct DShape {
    static constexpr int RC = R * C;
    // Blocks per chunk: up to 16 (one column per lane of a 16-lane row) and 64 weights (four
    // registers), more multiply-adds per chunk load than the per-lane layout's 32 weights; 1x1
    // keeps 8 (measured on MI355X, BERT-base FFN at 4096 tokens: 16-block chunks split its rows
    // of about 77 blocks unevenly between the two halves and ran 1.6 times longer, while 1x32,
    // 4x4 and 8x1 ran 7-20% faster with the larger chunks).
    static constexpr int U = RC == 1 ? 8 : (64 / RC >= 16 ? 16 : (64 / RC < 1 ? 1 : 64 / RC));
    static constexpr int NWORDS = U * RC;
    static constexpr int NWV = (NWORDS + 15) / 16;   // weight registers
    static constexpr int VW = VShape<R, C>::VW;
    static_assert(U <= 16 && NWORDS <= 64, "a chunk's columns fit one 16-lane row");
};

// Blocks per chunk of the kernels (per-lane or broadcast weights).
template <int R, int C, bool BF>
constexpr int kUnits = BF ? VShape<R, C>::U : DShape<R, C>::U;

template <int R, int C>
struct DOps {
    int j;                        // column of block (lane % 16) of the half's chunk
    float w[DShape<R, C>::NWV];   // word 16 k + lane % 16 of the half's chunk
};

// The chunk that starts `o` blocks into the row (ranges and offsets as in vload: past the
// row's end a load returns 0 and touches no memory).  Lane l reads word 16 k + l % 16 of the
// chunk's weights and column l % 16 of its blocks; lanes past the chunk read the next blocks'
// words, which no broadcast selects.
template <int R, int C>
__device__ __forceinline__ void dload(DOps<R, C> &ops, __amdgpu_buffer_rsrc_t ri,
                                      __amdgpu_buffer_rsrc_t rd, int o) {
    using S = DShape<R, C>;
    const int i = threadIdx.x & 15;
    ops.j = int(__builtin_amdgcn_raw_buffer_load_b32(ri, (o + i) * 4, 0, 0));
#pragma unroll
    for (int k = 0; k < DShape<R, C>::NWV; ++k)
        ops.w[k] = __uint_as_float(
            __builtin_amdgcn_raw_buffer_load_b32(rd, (o * S::RC + 16 * k + i) * 4, 0, 0));
}

// acc += w * x with w the value of lane L (0 .. 15, a constant once the caller's loops are
// unrolled) of acc's 16-lane row in register w.  The s_nop keeps two wait states between any
// vector-ALU write of w (a register copy the compiler may place just before) and its DPP read,
// which the compiler's hazard checks do not see inside the asm.
#define BSR_FMAC_BCAST(N)                                                                    \
    case N:                                                                                  \
        if (nop)                                                                             \
            asm("s_nop 1\n\tv_fmac_f32_dpp %0, %1, %2 row_newbcast:" #N                      \
                " row_mask:0xf bank_mask:0xf"                                                 \
                : "+v"(acc)                                                                  \
                : "v"(w), "v"(x));                                                           \
        else                                                                                 \
            asm("v_fmac_f32_dpp %0, %1, %2 row_newbcast:" #N " row_mask:0xf bank_mask:0xf"     \
                : "+v"(acc)                                                                  \
                : "v"(w), "v"(x));                                                           \
        break;
// `nop`: the first read of w in a chunk (the point after which the compiler has no reason to
// copy w again) carries the wait states; later reads of the same register follow it.
__device__ __forceinline__ void fmac_bcast(float &acc, float w, float x, int L, bool nop) {
    switch (L) {
        BSR_FMAC_BCAST(0) BSR_FMAC_BCAST(1) BSR_FMAC_BCAST(2) BSR_FMAC_BCAST(3)
        BSR_FMAC_BCAST(4) BSR_FMAC_BCAST(5) BSR_FMAC_BCAST(6) BSR_FMAC_BCAST(7)
        BSR_FMAC_BCAST(8) BSR_FMAC_BCAST(9) BSR_FMAC_BCAST(10) BSR_FMAC_BCAST(11)
        BSR_FMAC_BCAST(12) BSR_FMAC_BCAST(13) BSR_FMAC_BCAST(14) BSR_FMAC_BCAST(15)
        default: break;
    }
}
#undef BSR_FMAC_BCAST

// Lane L (0 .. 15, constant after unrolling) of v's 16-lane row, in every lane of the row.
#define BSR_BCAST(N) \
    case N: return __builtin_amdgcn_update_dpp(0, v, 0x150 + N, 0xf, 0xf, false);
__device__ __forceinline__ int bcast_lane(int v, int L) {
    switch (L) {
        BSR_BCAST(0) BSR_BCAST(1) BSR_BCAST(2) BSR_BCAST(3) BSR_BCAST(4) BSR_BCAST(5)
        BSR_BCAST(6) BSR_BCAST(7) BSR_BCAST(8) BSR_BCAST(9) BSR_BCAST(10) BSR_BCAST(11)
        BSR_BCAST(12) BSR_BCAST(13) BSR_BCAST(14) BSR_BCAST(15)
        default: return v;
    }
}
#undef BSR_BCAST

// base + (lane L of v's 16-lane row), one v_add_u32 with a DPP row broadcast of v (L constant
// after unrolling; `nop` on the first read of v after the vector-ALU op that wrote it, as for
// fmac_bcast).
#define BSR_ADD_BCAST(N)                                                                     \
    case N:                                                                                  \
        if (nop)                                                                             \
            asm("s_nop 1\n\tv_add_u32_dpp %0, %1, %2 row_newbcast:" #N                       \
                " row_mask:0xf bank_mask:0xf"                                                 \
                : "=v"(r)                                                                    \
                : "v"(v), "v"(base));                                                        \
        else                                                                                 \
            asm("v_add_u32_dpp %0, %1, %2 row_newbcast:" #N " row_mask:0xf bank_mask:0xf"      \
                : "=v"(r)                                                                    \
                : "v"(v), "v"(base));                                                        \
        break;
__device__ __forceinline__ unsigned add_bcast(unsigned v, unsigned base, int L, bool nop) {
    unsigned r = 0;
    switch (L) {
        BSR_ADD_BCAST(0) BSR_ADD_BCAST(1) BSR_ADD_BCAST(2) BSR_ADD_BCAST(3) BSR_ADD_BCAST(4)
        BSR_ADD_BCAST(5) BSR_ADD_BCAST(6) BSR_ADD_BCAST(7) BSR_ADD_BCAST(8) BSR_ADD_BCAST(9)
        BSR_ADD_BCAST(10) BSR_ADD_BCAST(11) BSR_ADD_BCAST(12) BSR_ADD_BCAST(13)
        BSR_ADD_BCAST(14) BSR_ADD_BCAST(15)
        default: break;
    }
    return r;
}
#undef BSR_ADD_BCAST

typedef __attribute__((address_space(3))) const float lds_cfloat;

// vcompute with broadcast operands: acc[r] += sum over the chunk's first nv blocks (all U when
// !MASKED) of X[t][j * C + c] * w[r][c], in the same order as vcompute (block, column, output
// row), so the sums are bitwise those of vcompute.  Each lane clamps and scales the column of
// its own block of the chunk once; a block's LDS address is then one broadcast add.
template <int R, int C, bool MASKED>
__device__ __forceinline__ void dcompute(float (&acc)[R], const DOps<R, C> &ops,
                                         const float *xrow, int Kb, int nv, int jlo = 0) {
    using S = DShape<R, C>;
    using V = typename VecOf<S::VW>::type;
    typedef __attribute__((address_space(3))) const V lds_cv;
    const unsigned xbase = unsigned(size_t((lds_cfloat *)xrow));   // its LDS byte address
    const unsigned cbytes = min(unsigned(ops.j - jlo), unsigned(Kb - 1)) * unsigned(C * 4);
    if constexpr (!MASKED && C == 1) {
        // One LDS read per block: issue the chunk's U reads before its first multiply-add, so
        // all of them are in flight at once (left to the scheduler, the reads and multiply-adds
        // interleaved with two or three reads outstanding, and the waves waited on LDS latency).
        float xs[S::U];
#pragma unroll
        for (int u = 0; u < S::U; ++u)
            xs[u] = *(lds_cfloat *)size_t(add_bcast(cbytes, xbase, u, u == 0));
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < S::U; ++u) {
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const int word = u * S::RC + r;
                fmac_bcast(acc[r], ops.w[word / 16], xs[u], word % 16, word % 16 == 0);
            }
        }
        return;
    }
    // A guard rather than a break: the loop keeps a constant trip count, so it unrolls fully
    // and every broadcast lane and weight register is a constant (with a break, chunks of 16
    // blocks were left rolled, with the weights in scratch memory and a switch per broadcast).
    // The guard is uniform over each 16-lane row (both rows of a half share nv).
#pragma unroll
    for (int u = 0; u < S::U; ++u) {
        if (!MASKED || u < nv) {
            const unsigned a = add_bcast(cbytes, xbase, u, u == 0);
#pragma unroll
            for (int c0 = 0; c0 < C; c0 += S::VW) {
                const V xv = *(lds_cv *)size_t(a + 4 * c0);
#pragma unroll
                for (int cc = 0; cc < S::VW; ++cc) {
                    float x;
                    if constexpr (S::VW == 1) x = xv;
                    else x = xv[cc];
#pragma unroll
                    for (int r = 0; r < R; ++r) {
                        const int word = u * S::RC + r * C + c0 + cc;
                        fmac_bcast(acc[r], ops.w[word / 16], x, word % 16, word % 16 == 0);
                    }
                }
            }
        }
    }
}

// A chunk's operands and their use: broadcast operands for fp32 weights, per-lane copies for
// bf16 weights (widening a bf16 weight is a vector-ALU write, which the broadcast's DPP read
// must not follow too closely).
template <int R, int C, bool BF>
using OpsOf = std::conditional_t<BF, VOps<R, C>, DOps<R, C>>;

template <int R, int C, bool BF>
__device__ __forceinline__ void oload(OpsOf<R, C, BF> &ops, __amdgpu_buffer_rsrc_t ri,
                                      __amdgpu_buffer_rsrc_t rd, int o) {
    if constexpr (BF) vload<R, C, BF>(ops, ri, rd, o);
    else dload<R, C>(ops, ri, rd, o);
}

template <int R, int C, bool BF, bool MASKED>
__device__ __forceinline__ void ocompute(float (&acc)[R], const OpsOf<R, C, BF> &ops,
                                         const float *xrow, int Kb, int nv, int jlo = 0) {
    if constexpr (BF) vcompute<R, C, MASKED>(acc, ops, xrow, Kb, nv, jlo);
    else dcompute<R, C, MASKED>(acc, ops, xrow, Kb, nv, jlo);
}

// The rows of a wave (fp32 weights) as one stream.  A wave's rows row0, row0 + step, ... are
// taken 64 at a time: lane k loads the row pointers and biases of row k of the group, then the
// wave walks the group's iterations (a row of nq chunks takes max(1, ceil(nq / 2)) of them; in
// iteration i of a row, half h multiplies chunk 2 i + h) as one sequence, with the operands of
// the next kDD iterations in flight.  Loads run ahead across row ends, so a row's first chunks
// arrive under the previous row's work; every phase issues one iteration's loads (past the
// group's last row they fetch nothing), so the waits count them.  A row's sums are those of
// the row loop (same chunks, same order).
constexpr int kDD = 8;
constexpr int kStreamRowsPerWave = 16;

// Lane k's value of v (k uniform), bit for bit.
__device__ __forceinline__ float lane_float(float v, int k) {
    return __uint_as_float(unsigned(__builtin_amdgcn_readlane(int(__float_as_uint(v)), k)));
}

template <int R, int C>
__device__ __forceinline__ void stream_rows(int row0, int row_hi, int step,
                                            const int32_t *__restrict__ indptr,
                                            const int32_t *__restrict__ indices,
                                            const void *__restrict__ data, int nnzb,
                                            const float *xrow, int Kb,
                                            __amdgpu_buffer_rsrc_t rb, __amdgpu_buffer_rsrc_t ry,
                                            int vo_row, int h) {
    using S = DShape<R, C>;
    constexpr int U = S::U;
    const int lane = threadIdx.x & 63;
    const __amdgpu_buffer_rsrc_t rip = buffer_rsrc(indptr, unsigned(row_hi + 1) * 4u);
#pragma unroll 1
    for (int g0 = row0; g0 < row_hi; g0 += 64 * step) {
        // The group: rows g0 + step k, k < nr.
        const int nr = min(64, (row_hi - g0 + step - 1) / step);
        int ip0, ip1;
        float bv[R];
        {
            const int row = g0 + step * (lane < nr ? lane : 0);
            const int a = int(__builtin_amdgcn_raw_buffer_load_b32(rip, row * 4, 0, 0));
            const int b = int(__builtin_amdgcn_raw_buffer_load_b32(rip, row * 4 + 4, 0, 0));
            ip0 = clampi(a, 0, nnzb);
            ip1 = clampi(b, ip0, nnzb);
#pragma unroll
            for (int r = 0; r < R; ++r)
                bv[r] = __uint_as_float(
                    __builtin_amdgcn_raw_buffer_load_b32(rb, (row * R + r) * 4, 0, 0));
        }
        // Load cursor: row kl of the group, its iteration il, and the row's operand ranges.
        int kl = 0, il = 0, lp0 = 0, lm = 0, lits = 0;
        __amdgpu_buffer_rsrc_t ri = buffer_rsrc(indices, 0u), rd = buffer_rsrc(data, 0u);
        auto open_row = [&]() {   // kl < nr
            lp0 = __builtin_amdgcn_readlane(ip0, kl);
            lm = __builtin_amdgcn_readlane(ip1, kl) - lp0;
            const int nq = (lm + U - 1) / U;
            lits = nq > 2 ? (nq + 1) >> 1 : 1;
            ri = buffer_rsrc(indices + lp0, unsigned(lm) * 4u);
            rd = buffer_rsrc(static_cast<const float *>(data) + int64_t(lp0) * S::RC,
                             unsigned(lm) * unsigned(S::RC * 4));
        };
        open_row();
        auto load_next = [&](DOps<R, C> &o) {
            // Iteration il of row kl (nothing once the group is done), then advance.
            if (kl < nr) {
                dload<R, C>(o, ri, rd, (2 * il + h) * U);
                if (++il == lits) {
                    il = 0;
                    if (++kl < nr) open_row();
                }
            } else {
                const __amdgpu_buffer_rsrc_t z = buffer_rsrc(indices, 0u);
                dload<R, C>(o, z, z, 0);
            }
        };
        DOps<R, C> ring[kDD];
#pragma unroll
        for (int d = 0; d < kDD; ++d) load_next(ring[d]);
        // Compute cursor: row kc, its iteration ic and iteration count.
        int kc = 0, ic = 0;
        int cm = __builtin_amdgcn_readlane(ip1, 0) - __builtin_amdgcn_readlane(ip0, 0);
        int cits;
        {
            const int nq = (cm + U - 1) / U;
            cits = nq > 2 ? (nq + 1) >> 1 : 1;
        }
        float acc[R];
#pragma unroll
        for (int r = 0; r < R; ++r) acc[r] = h == 0 ? lane_float(bv[r], 0) : 0.0f;
#pragma unroll 1
        while (kc < nr) {
#pragma unroll
            for (int ph = 0; ph < kDD; ++ph) {
                if (kc < nr) {
                    const int nv = cm - (2 * ic + h) * U;
                    if (ic + 1 == cits) {
                        dcompute<R, C, true>(acc, ring[ph], xrow, Kb, nv);
                        // Row kc is complete: sum the halves (as in the row loop) and store.
                        const int n0 = (g0 + step * kc) * R;
                        const int vo = vo_row + n0 * 4;
                        constexpr int kHalf = R == 1 ? 1 : R / 2;
#pragma unroll
                        for (int r = 0; r < kHalf; ++r) {
                            const float P = acc[r], Q = acc[R == 1 ? 0 : R / 2 + r];
                            const auto sw = __builtin_amdgcn_permlane32_swap(
                                __float_as_uint(P), __float_as_uint(Q), false, false);
                            const float y = __uint_as_float(sw[0]) + __uint_as_float(sw[1]);
                            if (R > 1 || h == 0)
                                __builtin_amdgcn_raw_buffer_store_b32(
                                    __float_as_uint(y), ry, vo + (h * kHalf + r) * 4 * (R > 1),
                                    0, 0);
                        }
                        ++kc;
                        ic = 0;
                        if (kc < nr) {
                            const int a = __builtin_amdgcn_readlane(ip0, kc);
                            cm = __builtin_amdgcn_readlane(ip1, kc) - a;
                            const int nq = (cm + U - 1) / U;
                            cits = nq > 2 ? (nq + 1) >> 1 : 1;
#pragma unroll
                            for (int r = 0; r < R; ++r)
                                acc[r] = h == 0 ? lane_float(bv[r], kc) : 0.0f;
                        }
                    } else {
                        dcompute<R, C, false>(acc, ring[ph], xrow, Kb, U);
                        ++ic;
                    }
                }
                __builtin_amdgcn_sched_barrier(0);
                load_next(ring[ph]);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    }
}

template <int R, int C, bool BF>
__global__ __launch_bounds__((kWaves<R, C, BF> * 64)) void spmm_vtile_kernel(const TiledBatch batch) {
    using S = VShape<R, C>;
    constexpr int NW = kWaves<R, C, BF>, U = kUnits<R, C, BF>;
    extern __shared__ float smem[];
    float *Xs = smem;

    const int lane = threadIdx.x & 63, wave = uniform(threadIdx.x >> 6);
    const int t = lane & 31, h = lane >> 5;

    const TiledItem &I = batch.item[blockIdx.y];
    const void *__restrict__ X = I.X;
    const int64_t T = I.T, ldx = I.ldx, ldy = I.ldy;
    const int32_t *__restrict__ indptr = I.indptr;
    const int32_t *__restrict__ indices = I.indices;
    const void *__restrict__ data = I.data;
    const float *__restrict__ bias = I.bias;
    float *__restrict__ Y = I.Y;
    const int K = I.K, nnzb = I.nnzb, Nb = I.Nb, Kb = I.Kb, num_tiles = I.num_tiles,
              slices = I.slices, XP = I.XP;

    // Workgroup -> (token tile, slice): workgroups are dealt to the 8 XCDs round robin (the
    // grid's x extent is a multiple of 8), and the product's (tile, slice) pairs, tile-major,
    // are cut into 8 contiguous ranges, one per XCD, so a tile's slices share few L2s.
    const int g = blockIdx.x, xcd = g & 7, rank = g >> 3;
    const int pairs = num_tiles * slices, per_xcd = (pairs + 7) >> 3;
    const int q = xcd * per_xcd + rank;
    if (rank >= per_xcd || q >= pairs) return;
    const int tile = q / slices, s = q - tile * slices;
    const int64_t t0 = int64_t(tile) * kVT;
    const int rows = int(T - t0 < kVT ? T - t0 : kVT);
    const int row_lo = int(int64_t(s) * Nb / slices), row_hi = int(int64_t(s + 1) * Nb / slices);

    // Stage X[t0 : t0 + 32][0 : K] as fp32, row pitch XP.  Each wave moves whole rows, eight
    // 64-column groups of loads in flight before their LDS stores; rows past T read as 0 (an
    // empty buffer range).
    {
        constexpr int kXBytes = BF ? 2 : 4;
        constexpr int kG = 8;
#pragma unroll 1
        for (int tr = wave; tr < kVT; tr += NW) {
            const int src = tr < rows ? tr : 0;
            const __amdgpu_buffer_rsrc_t rx =
                buffer_rsrc(static_cast<const char *>(X) + (t0 + src) * ldx * kXBytes,
                            tr < rows ? unsigned(K) * kXBytes : 0u);
            float *dst = Xs + tr * XP;
            float *spare = Xs + kVT * XP + lane;
#pragma unroll 1
            for (int c0 = 0; c0 < K; c0 += 64 * kG) {
                float v[kG];
#pragma unroll
                for (int m = 0; m < kG; ++m) {
                    const int c = c0 + 64 * m + lane;
                    if constexpr (BF)
                        v[m] = __uint_as_float(unsigned(__builtin_amdgcn_raw_buffer_load_b16(
                                                   rx, c * 2, 0, 0))
                                               << 16);
                    else
                        v[m] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rx, c * 4, 0, 0));
                }
                // Branch-free stores: a lane past the end of the row writes its word of the
                // spare region after the tile, which nothing reads.
#pragma unroll
                for (int m = 0; m < kG; ++m) {
                    const int c = c0 + 64 * m + lane;
                    *(c < K ? dst + c : spare) = v[m];
                }
            }
        }
    }
    __syncthreads();

    const float *xrow = Xs + t * XP;
    const int ldy4 = int(ldy) * 4;
    const __amdgpu_buffer_rsrc_t ry =
        buffer_rsrc(Y + t0 * ldy, unsigned(rows) * unsigned(ldy4));
    const __amdgpu_buffer_rsrc_t rb = buffer_rsrc(bias, bias ? unsigned(Nb * R) * 4u : 0u);
    constexpr int kEs = BF ? 2 : 4;   // bytes per stored weight

    if constexpr (!BF) {
        // Many rows per wave: the streamed loop (its prologue per 64 rows costs more than it
        // saves on short slices: measured slower at 2 and 12 rows per wave, faster at 24+).
        if (row_hi - row_lo >= kStreamRowsPerWave * NW) {
            stream_rows<R, C>(row_lo + wave, row_hi, NW, indptr, indices, data, nnzb, xrow, Kb,
                              rb, ry, t * ldy4, h);
            return;
        }
    }

#pragma unroll 1
    for (int row = row_lo + wave; row < row_hi; row += NW) {
        const int p0 = clampi(uniform(indptr[row]), 0, nnzb);
        const int p1 = clampi(uniform(indptr[row + 1]), p0, nnzb);
        const int m = p1 - p0;
        const int n0 = row * R;
        float acc[R];
        // Half 0 starts from the bias (a NULL bias reads 0), half 1 from zero.
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const float b = __uint_as_float(
                __builtin_amdgcn_raw_buffer_load_b32(rb, (n0 + r) * 4, 0, 0));
            acc[r] = h == 0 ? b : 0.0f;
        }
        if (m > 0) {
            const __amdgpu_buffer_rsrc_t ri = buffer_rsrc(indices + p0, unsigned(m) * 4u);
            const __amdgpu_buffer_rsrc_t rd = buffer_rsrc(
                static_cast<const char *>(data) + int64_t(p0) * S::RC * kEs,
                unsigned(m) * unsigned(S::RC * kEs));
            const int nq = (m + U - 1) / U, iters = (nq + 1) >> 1;
            // Chunk `it` of this half starts (2 it + h) U blocks into the row; every chunk
            // before the last iteration is full.  The next chunk is loaded in every iteration,
            // also past the row's end (those loads return 0 and touch no memory), so the wait
            // for the current chunk always leaves the next one's loads in flight (a conditional
            // load left the compiler's wait at zero outstanding loads).
            OpsOf<R, C, BF> A, B;
            oload<R, C, BF>(A, ri, rd, h * U);
            int it = 0;
            while (true) {
                oload<R, C, BF>(B, ri, rd, (2 * (it + 1) + h) * U);
                __builtin_amdgcn_sched_barrier(0);
                if (it + 1 >= iters) {
                    ocompute<R, C, BF, true>(acc, A, xrow, Kb, m - (2 * it + h) * U);
                    break;
                }
                ocompute<R, C, BF, false>(acc, A, xrow, Kb, U);
                __builtin_amdgcn_sched_barrier(0);
                ++it;
                oload<R, C, BF>(A, ri, rd, (2 * (it + 1) + h) * U);
                __builtin_amdgcn_sched_barrier(0);
                if (it + 1 >= iters) {
                    ocompute<R, C, BF, true>(acc, B, xrow, Kb, m - (2 * it + h) * U);
                    break;
                }
                ocompute<R, C, BF, false>(acc, B, xrow, Kb, U);
                __builtin_amdgcn_sched_barrier(0);
                ++it;
            }
        }
        // Sum the halves and store.  v_permlane32_swap(P, Q) exchanges the upper half of P
        // with the lower half of Q, giving P' = [P_lo | Q_lo] and Q' = [P_hi | Q_hi]; so with
        // P = acc[r] and Q = acc[R/2 + r], P' + Q' is the total of output r on half 0 and of
        // output R/2 + r on half 1, both summed as (half 0) + (half 1).  Half h then stores
        // outputs [h R/2, (h+1) R/2) of its token (R = 1: P = Q, and half 0 stores).
        const int vo = t * ldy4 + n0 * 4;
        constexpr int kHalf = R == 1 ? 1 : R / 2;
        static_assert(R == 1 || R % 2 == 0, "two-half stores need an even R");
#pragma unroll
        for (int r = 0; r < kHalf; ++r) {
            const float P = acc[r], Q = acc[R == 1 ? 0 : R / 2 + r];
            const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(P),
                                                             __float_as_uint(Q), false, false);
            const float y = __uint_as_float(sw[0]) + __uint_as_float(sw[1]);
            if (R > 1 || h == 0)
                __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(y), ry,
                                                      vo + (h * kHalf + r) * 4 * (R > 1), 0, 0);
        }
    }
}

// ---------------------------------------------------------------- column-chunked variant
// Inputs too wide for one LDS X tile (e.g. the 3072-column input of BERT's FFN output layer):
// the same lanes, chunks of U blocks and two halves per row as above, with the input columns
// cut into chunks of chunk_blocks block-columns as in the column-chunked matrix-core kernel.
// Each wave owns up to VChunkRows<R> rows of the slice (row_lo + wave + NW i) and keeps their
// accumulators in registers from the first chunk to the last; per chunk it stages the chunk's
// columns of the X tile, finds where each of its rows leaves the chunk (indices ascend within
// a row: the first index at or past the chunk's end, by ballots over 256 indices at a time)
// and runs the row's blocks up to there.  Rows are stored once, after the last chunk.
template <int R>
struct VChunkRows {
    static constexpr int value = R == 1 ? 8 : (R <= 4 ? 4 : 2);
};

template <int R, int C, bool BF>
__global__ __launch_bounds__((kWaves<R, C, BF> * 64)) void spmm_vtile_chunk_kernel(
    const KchunkBatch batch) {
    using S = VShape<R, C>;
    constexpr int NW = kWaves<R, C, BF>, U = kUnits<R, C, BF>, MR = VChunkRows<R>::value;
    extern __shared__ float smem[];
    float *Xs = smem;

    const int lane = threadIdx.x & 63, wave = uniform(threadIdx.x >> 6);
    const int t = lane & 31, h = lane >> 5;

    const KchunkItem &I = batch.item[blockIdx.y];
    const void *__restrict__ X = I.X;
    const int64_t T = I.T, ldx = I.ldx, ldy = I.ldy;
    const int32_t *__restrict__ indptr = I.indptr;
    const int32_t *__restrict__ indices = I.indices;
    const void *__restrict__ data = I.data;
    const float *__restrict__ bias = I.bias;
    float *__restrict__ Y = I.Y;
    const int nnzb = I.nnzb, Nb = I.Nb, Kb = I.Kb, num_tiles = I.num_tiles,
              slices = I.slices, XP = I.XP, kcb = I.chunk_blocks, nchunks = I.nchunks;

    const int g = blockIdx.x, xcd = g & 7, rank = g >> 3;
    const int pairs = num_tiles * slices, per_xcd = (pairs + 7) >> 3;
    const int q = xcd * per_xcd + rank;
    if (rank >= per_xcd || q >= pairs) return;
    const int tile = q / slices, s = q - tile * slices;
    const int64_t t0 = int64_t(tile) * kVT;
    const int rows = int(T - t0 < kVT ? T - t0 : kVT);
    const int row_lo = int(int64_t(s) * Nb / slices), row_hi = int(int64_t(s + 1) * Nb / slices);

    // This wave's rows, their block ranges [pos, end) and accumulators (half 0 starts from the
    // bias, half 1 from zero).
    const __amdgpu_buffer_rsrc_t rb = buffer_rsrc(bias, bias ? unsigned(Nb * R) * 4u : 0u);
    int pos[MR], end[MR];
    float acc[MR][R];
#pragma unroll
    for (int i = 0; i < MR; ++i) {
        const int row = row_lo + wave + NW * i;
        pos[i] = end[i] = 0;
        if (row < row_hi) {
            pos[i] = clampi(uniform(indptr[row]), 0, nnzb);
            end[i] = clampi(uniform(indptr[row + 1]), pos[i], nnzb);
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const float b = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
                rb, (row < row_hi ? row * R + r : 0) * 4, 0, 0));
            acc[i][r] = h == 0 && row < row_hi ? b : 0.0f;
        }
    }

    // First position in [p, e) whose block column is >= jhi, else e.
    auto crossing = [&](int p, int e, int jhi) -> int {
        for (int base = p; base < e; base += 256) {
            const __amdgpu_buffer_rsrc_t ri =
                buffer_rsrc(indices + base, unsigned(e - base) * 4u);
            int x[4];
#pragma unroll
            for (int m = 0; m < 4; ++m)
                x[m] = __builtin_amdgcn_raw_buffer_load_b32(ri, (lane + 64 * m) * 4, 0, 0);
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                const unsigned long long b = __ballot(base + 64 * m + lane < e && x[m] >= jhi);
                if (b) return base + 64 * m + __ffsll(static_cast<long long>(b)) - 1;
            }
        }
        return e;
    };

    const float *xrow = Xs + t * XP;
    constexpr int kEs = BF ? 2 : 4;   // bytes per stored weight
    for (int c = 0; c < nchunks; ++c) {
        const int jlo = c * kcb;
        const int jhi = c + 1 == nchunks ? Kb : jlo + kcb;
        const int kbw = jhi - jlo, cols = kbw * C;
        if (c > 0) __syncthreads();   // every wave is done with the previous chunk's tile
        // Stage X[t0 : t0 + 32][jlo*C : jlo*C + cols] as fp32, row pitch XP (as above).
        {
            constexpr int kXBytes = BF ? 2 : 4;
            constexpr int kG = 8;
#pragma unroll 1
            for (int tr = wave; tr < kVT; tr += NW) {
                const int src = tr < rows ? tr : 0;
                const __amdgpu_buffer_rsrc_t rx = buffer_rsrc(
                    static_cast<const char *>(X) + ((t0 + src) * ldx + int64_t(jlo) * C) * kXBytes,
                    tr < rows ? unsigned(cols) * kXBytes : 0u);
                float *dst = Xs + tr * XP;
                float *spare = Xs + kVT * XP + lane;
#pragma unroll 1
                for (int c0 = 0; c0 < cols; c0 += 64 * kG) {
                    float v[kG];
#pragma unroll
                    for (int m = 0; m < kG; ++m) {
                        const int cc = c0 + 64 * m + lane;
                        if constexpr (BF)
                            v[m] = __uint_as_float(unsigned(__builtin_amdgcn_raw_buffer_load_b16(
                                                       rx, cc * 2, 0, 0))
                                                   << 16);
                        else
                            v[m] = __uint_as_float(
                                __builtin_amdgcn_raw_buffer_load_b32(rx, cc * 4, 0, 0));
                    }
#pragma unroll
                    for (int m = 0; m < kG; ++m) {
                        const int cc = c0 + 64 * m + lane;
                        *(cc < cols ? dst + cc : spare) = v[m];
                    }
                }
            }
        }
        int cend[MR];
#pragma unroll
        for (int i = 0; i < MR; ++i)
            cend[i] = c + 1 == nchunks ? end[i] : crossing(pos[i], end[i], jhi);
        __syncthreads();

#pragma unroll
        for (int i = 0; i < MR; ++i) {
            const int p0 = pos[i], m = cend[i] - pos[i];
            pos[i] = cend[i];
            if (m <= 0) continue;
            const __amdgpu_buffer_rsrc_t ri = buffer_rsrc(indices + p0, unsigned(m) * 4u);
            const __amdgpu_buffer_rsrc_t rd = buffer_rsrc(
                static_cast<const char *>(data) + int64_t(p0) * S::RC * kEs,
                unsigned(m) * unsigned(S::RC * kEs));
            const int nq = (m + U - 1) / U, iters = (nq + 1) >> 1;
            OpsOf<R, C, BF> A, B;
            oload<R, C, BF>(A, ri, rd, h * U);
            int it = 0;
            while (true) {
                oload<R, C, BF>(B, ri, rd, (2 * (it + 1) + h) * U);
                __builtin_amdgcn_sched_barrier(0);
                if (it + 1 >= iters) {
                    ocompute<R, C, BF, true>(acc[i], A, xrow, kbw, m - (2 * it + h) * U, jlo);
                    break;
                }
                ocompute<R, C, BF, false>(acc[i], A, xrow, kbw, U, jlo);
                __builtin_amdgcn_sched_barrier(0);
                ++it;
                oload<R, C, BF>(A, ri, rd, (2 * (it + 1) + h) * U);
                __builtin_amdgcn_sched_barrier(0);
                if (it + 1 >= iters) {
                    ocompute<R, C, BF, true>(acc[i], B, xrow, kbw, m - (2 * it + h) * U, jlo);
                    break;
                }
                ocompute<R, C, BF, false>(acc[i], B, xrow, kbw, U, jlo);
                __builtin_amdgcn_sched_barrier(0);
                ++it;
            }
        }
    }

    // Sum the halves and store, as above.
    const int ldy4 = int(ldy) * 4;
    const __amdgpu_buffer_rsrc_t ry = buffer_rsrc(Y + t0 * ldy, unsigned(rows) * unsigned(ldy4));
    constexpr int kHalf = R == 1 ? 1 : R / 2;
#pragma unroll
    for (int i = 0; i < MR; ++i) {
        const int row = row_lo + wave + NW * i;
        if (row >= row_hi) continue;
        const int vo = t * ldy4 + row * R * 4;
#pragma unroll
        for (int r = 0; r < kHalf; ++r) {
            const float P = acc[i][r], Q = acc[i][R == 1 ? 0 : R / 2 + r];
            const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(P),
                                                             __float_as_uint(Q), false, false);
            const float y = __uint_as_float(sw[0]) + __uint_as_float(sw[1]);
            if (R > 1 || h == 0)
                __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(y), ry,
                                                      vo + (h * kHalf + r) * 4 * (R > 1), 0, 0);
        }
    }
}

template <int R, int C, bool BF>
bsr_status launch_vchunk_variant(const KchunkBatch &batch, dim3 grid, size_t lds, hipStream_t st,
                                 const LaunchEvents &ev) {
    launch_kernel(spmm_vtile_chunk_kernel<R, C, BF>, grid, dim3(kWaves<R, C, BF> * 64), lds, st,
                  ev, batch);
    return launch_status();
}

template <bool BF>
bsr_status launch_vchunk_shape(int R, int C, const KchunkBatch &b, dim3 g, size_t lds,
                               hipStream_t st, const LaunchEvents &ev) {
#define BSR_VCHUNK(RR, CC) \
    if (R == RR && C == CC) return launch_vchunk_variant<RR, CC, BF>(b, g, lds, st, ev);
    if constexpr (!BF) {
        BSR_VCHUNK(1, 1)
    }
    BSR_VCHUNK(1, 2)
    BSR_VCHUNK(1, 4)
    BSR_VCHUNK(1, 8)
    BSR_VCHUNK(1, 16)
    BSR_VCHUNK(1, 32)
    BSR_VCHUNK(2, 1)
    BSR_VCHUNK(4, 1)
    BSR_VCHUNK(8, 1)
    BSR_VCHUNK(2, 2)
    BSR_VCHUNK(4, 4)
    BSR_VCHUNK(8, 8)
#undef BSR_VCHUNK
    return BSR_ERR_UNSUPPORTED;
}

template <int R, int C, bool BF>
bsr_status launch_vtile_variant(const TiledBatch &batch, dim3 grid, size_t lds, hipStream_t st,
                                const LaunchEvents &ev) {
    launch_kernel(spmm_vtile_kernel<R, C, BF>, grid, dim3(kWaves<R, C, BF> * 64), lds, st, ev,
                  batch);
    return launch_status();
}

// The shapes instantiated here, for one dtype.
template <bool BF>
bsr_status launch_vtile_shape(int R, int C, const TiledBatch &b, dim3 g, size_t lds,
                              hipStream_t st, const LaunchEvents &ev) {
#define BSR_VTILE(RR, CC) \
    if (R == RR && C == CC) return launch_vtile_variant<RR, CC, BF>(b, g, lds, st, ev);
    if constexpr (!BF) {
        BSR_VTILE(1, 1)
    }
    BSR_VTILE(1, 2)
    BSR_VTILE(1, 4)
    BSR_VTILE(1, 8)
    BSR_VTILE(1, 16)
    BSR_VTILE(1, 32)
    BSR_VTILE(2, 1)
    BSR_VTILE(4, 1)
    BSR_VTILE(8, 1)
    BSR_VTILE(2, 2)
    BSR_VTILE(4, 4)
    BSR_VTILE(8, 8)
#undef BSR_VTILE
    return BSR_ERR_UNSUPPORTED;
}

}  // namespace

bool vtile_supported(int R, int C, int dtype) {
    if (dtype != BSR_F32 && dtype != BSR_BF16) return false;
    const bool shape = (R == 1 && (C == 1 || C == 2 || C == 4 || C == 8 || C == 16 || C == 32)) ||
                       (C == 1 && (R == 2 || R == 4 || R == 8)) ||
                       (R == C && (R == 2 || R == 4 || R == 8));
    // bf16 blocks of one element would start at 2-byte offsets; the loads want 4.
    return shape && !(dtype == BSR_BF16 && R * C == 1);
}

TiledPlan plan_vtile(const void *X, int64_t T, int64_t ldx, const bsr_matrix_t *W, int64_t ldy,
                     int slices, size_t lds_limit) {
    TiledPlan p{};
    const int R = W->R, C = W->C;
    if (!vtile_supported(R, C, W->dtype)) return p;
    const int64_t K = W->n_cols, Nb = W->n_rows / R;
    // Row pitch XP >= K with XP = VW (mod 2 VW): reads of VW floats by consecutive tokens
    // start VW banks apart (mod 2 VW), so a column segment read by 32 tokens is conflict-free.
    const int vw = C % 4 == 0 ? 4 : (C % 2 == 0 ? 2 : 1);
    const int64_t xp = K + (((vw - K) % (2 * vw)) + 2 * vw) % (2 * vw);
    p.x_pitch = int(xp);
    p.lds_bytes = (size_t(kVT) * size_t(xp) + 64) * 4;   // the tile, then 64 spare words
    if (p.lds_bytes > lds_limit) return TiledPlan{};
    // 32-bit buffer ranges: the blocks of one row, one X row and a 32-row tile of Y.
    if (W->nnzb * R * C >= (int64_t(1) << 29)) return TiledPlan{};
    if (ldy >= (int64_t(1) << 24) || K >= (int64_t(1) << 24)) return TiledPlan{};
    p.num_tiles = int((T + kVT - 1) / kVT);
    p.slices = slices > 0 ? slices : 1;
    if (p.slices > Nb) p.slices = int(Nb);
    p.ok = true;
    return p;
}

bsr_status launch_spmm_vtile(const TiledWork *work, int n, void *stream,
                             const LaunchEvents &ev) {
    if (n < 1 || n > kMaxItems) return BSR_ERR_ARG;
    const int R = work[0].W->R, C = work[0].W->C, dtype = work[0].W->dtype;
    TiledBatch batch{};
    batch.n = n;
    int gx = 0;
    size_t lds = 0;
    for (int i = 0; i < n; ++i) {
        const TiledWork &w = work[i];
        if (w.W->R != R || w.W->C != C || w.W->dtype != dtype) return BSR_ERR_ARG;
        TiledItem &it = batch.item[i];
        it.X = w.X;
        it.T = w.T;
        it.ldx = w.ldx;
        it.indptr = w.W->indptr;
        it.indices = w.W->indices;
        it.data = w.W->data;
        it.bias = w.bias;
        it.Y = w.Y;
        it.ldy = w.ldy;
        it.K = int(w.W->n_cols);
        it.nnzb = int(w.W->nnzb);
        it.Nb = int(w.W->n_rows / R);
        it.Kb = int(w.W->n_cols / C);
        it.num_tiles = w.plan.num_tiles;
        it.slices = w.plan.slices;
        it.XP = w.plan.x_pitch;
        const int wgs = ((w.plan.num_tiles * w.plan.slices + 7) / 8) * 8;
        if (wgs > gx) gx = wgs;
        if (w.plan.lds_bytes > lds) lds = w.plan.lds_bytes;
    }
    hipStream_t st = as_stream(stream);
    const dim3 grid(gx, n);
    if (dtype == BSR_BF16) return launch_vtile_shape<true>(R, C, batch, grid, lds, st, ev);
    return launch_vtile_shape<false>(R, C, batch, grid, lds, st, ev);
}

KchunkPlan plan_vchunk(const void *X, int64_t T, int64_t ldx, const bsr_matrix_t *W,
                       int64_t ldy, int slices, size_t lds_limit) {
    KchunkPlan kp{};
    const int R = W->R, C = W->C;
    if (!vtile_supported(R, C, W->dtype)) return kp;
    const int64_t K = W->n_cols, Nb = W->n_rows / R, Kb = K / C;
    const int vw = C % 4 == 0 ? 4 : (C % 2 == 0 ? 2 : 1);
    // kWaves: 16 for fp32 weights, else VShape::NW.
    const int nw = W->dtype == BSR_F32
                       ? 16
                       : (R * C * (R * C >= 32 ? 1 : (32 / (R * C) > 8 ? 8 : 32 / (R * C))) <= 16
                              ? 16
                              : 8);
    const int mr = R == 1 ? 8 : (R <= 4 ? 4 : 2);   // VChunkRows<R>
    // Slices: at least enough that no wave owns more than mr rows.
    int64_t S = slices > 0 ? slices : 1;
    const int64_t min_s = (Nb + int64_t(nw) * mr - 1) / (int64_t(nw) * mr);
    if (S < min_s) S = min_s;
    if (S > Nb) S = Nb;
    // The widest chunk whose fp32 tile (pitch = width rounded up to VW mod 2 VW, plus the 64
    // spare words) fits.
    const int64_t words = int64_t(lds_limit) / 4 - 64;
    const int64_t cmax = words / kVT - 2 * vw;
    const int64_t kcb_max = cmax / C;
    if (kcb_max < 1) return KchunkPlan{};
    const int64_t nch = (Kb + kcb_max - 1) / kcb_max;
    const int64_t kcb = (Kb + nch - 1) / nch;
    const int64_t kc = kcb * C;
    TiledPlan &p = kp.base;
    p.x_pitch = int(kc + (((vw - kc) % (2 * vw)) + 2 * vw) % (2 * vw));
    p.lds_bytes = (size_t(kVT) * size_t(p.x_pitch) + 64) * 4;
    if (p.lds_bytes > lds_limit) return KchunkPlan{};
    if (W->nnzb * R * C >= (int64_t(1) << 29)) return KchunkPlan{};
    if (ldy >= (int64_t(1) << 24) || K >= (int64_t(1) << 24)) return KchunkPlan{};
    p.num_tiles = int((T + kVT - 1) / kVT);
    p.slices = int(S);
    p.ok = true;
    kp.chunk_blocks = int(kcb);
    kp.nchunks = int(nch);
    return kp;
}

bsr_status launch_spmm_vchunk(const KchunkWork *work, int n, void *stream,
                              const LaunchEvents &ev) {
    if (n < 1 || n > kMaxItems) return BSR_ERR_ARG;
    const int R = work[0].W->R, C = work[0].W->C, dtype = work[0].W->dtype;
    KchunkBatch batch{};
    batch.n = n;
    int gx = 0;
    size_t lds = 0;
    for (int i = 0; i < n; ++i) {
        const KchunkWork &w = work[i];
        if (w.W->R != R || w.W->C != C || w.W->dtype != dtype) return BSR_ERR_ARG;
        KchunkItem &it = batch.item[i];
        it.X = w.X;
        it.T = w.T;
        it.ldx = w.ldx;
        it.indptr = w.W->indptr;
        it.indices = w.W->indices;
        it.data = w.W->data;
        it.bias = w.bias;
        it.Y = w.Y;
        it.ldy = w.ldy;
        it.nnzb = int(w.W->nnzb);
        it.Nb = int(w.W->n_rows / R);
        it.Kb = int(w.W->n_cols / C);
        it.num_tiles = w.plan.base.num_tiles;
        it.slices = w.plan.base.slices;
        it.XP = w.plan.base.x_pitch;
        it.bias_words = 0;
        it.wbuf_offset = 0;
        it.chunk_blocks = w.plan.chunk_blocks;
        it.nchunks = w.plan.nchunks;
        const int wgs = ((w.plan.base.num_tiles * w.plan.base.slices + 7) / 8) * 8;
        if (wgs > gx) gx = wgs;
        if (w.plan.base.lds_bytes > lds) lds = w.plan.base.lds_bytes;
    }
    hipStream_t st = as_stream(stream);
    const dim3 grid(gx, n);
    if (dtype == BSR_BF16) return launch_vchunk_shape<true>(R, C, batch, grid, lds, st, ev);
    return launch_vchunk_shape<false>(R, C, batch, grid, lds, st, ev);
}

}  // namespace bsr
