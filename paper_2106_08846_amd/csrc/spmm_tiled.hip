// Tiled BSR product on gfx950 matrix cores (fp32 inputs, fp32 accumulate).
//
// Y[t][n] = bias[n] + sum over stored blocks p of block-row i = n / R of
//           sum over c < C of X[t][indices[p] * C + c] * data[p][n - iR][c]          (Sec. 2.2)
//
// For one block-row and a tile of tokens this is a small dense product once the input columns
// named by `indices` are gathered: Y_tile (tokens x R) += X_tile[:, cols] (tokens x m*C) times
// the row's blocks (m*C x R).  The kernels below run it on MFMA:
//
//   * R x 1 blocks (32x1, 16x1): the contraction index is the block.  32x1 uses
//     v_mfma_f32_32x32x2_f32 with two blocks per instruction; lane l supplies token l%32 of
//     block l/32 (gathered from the LDS X tile) and feature l%32 of that block's data, so the B
//     operand is one contiguous 256-byte load per instruction.  16x1 uses
//     v_mfma_f32_16x16x4_f32, four blocks per instruction, for two 16-token halves.
//   * R x R blocks (32x32, 16x16): the contraction index is the block column c.  Each lane
//     loads 16 contiguous bytes of the block (one float4 of a block row), and the order of c
//     inside each instruction is permuted identically for the A and B operands, which the sum
//     does not see.  A comes from the LDS X tile with 16-byte reads.
//
// Work decomposition (one workgroup = 32 tokens x one slice of block-rows):
//   * the X tile [32 tokens][K] is staged once into LDS, row pitch K+1 (R x 1: conflict-free
//     4-byte gathers of one column for 32 tokens) or K+4 (square blocks: 16-byte aligned rows);
//   * slices hold whole block-rows, balanced by stored-block count;
//   * inside a slice the stored blocks are split evenly over the waves (so skewed rows are
//     spread over several waves); a block-row cut by a wave boundary is summed by the wave where
//     it starts, adding the other waves' partial tiles from LDS in wave order after a barrier.
//     The summation order is fixed by the launch shape, so results are bitwise reproducible.
//   * workgroup ids are mapped so that the slices of one token tile run on the same XCD and
//     share its L2 for the X tile.
#include "device_common.h"
#include "spmm_tiled.h"

namespace bsr {

namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kTT = 32;  // tokens per workgroup

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

// ---------------------------------------------------------------------------------- engines
// Each engine knows its accumulator tile, how to add blocks [pa, pb) of one block-row into it,
// how to store it to Y (with bias), and how to spill / add it through LDS.

template <int R, int C>
struct Engine;

// 32x1 blocks, v_mfma_f32_32x32x2_f32.  acc[v] of lane l holds
// Y[t0 + 8*(v/4) + 4*(l/32) + v%4][n0 + l%32].
template <>
struct Engine<32, 1> {
    using Acc = floatx16;
    static constexpr int kRegs = 16;
    static constexpr int kPad = 1;
    __device__ static void zero(Acc &a) {
#pragma unroll
        for (int v = 0; v < 16; ++v) a[v] = 0.0f;
    }
    __device__ static void accumulate(Acc &acc, int pa, int pb, const int *__restrict__ indices,
                                      const float *__restrict__ data, const float *Xs, int XP,
                                      int Kb) {
        const int lane = threadIdx.x & 63, tl = lane & 31, kh = lane >> 5;
        const float *xrow = Xs + tl * XP;
        int p = pa;
        for (; p + 8 <= pb; p += 8) {
            int j[4];
            float b[4], a[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int q = p + 2 * u + kh;
                j[u] = clampi(indices[q], 0, Kb - 1);
                b[u] = data[int64_t(q) * 32 + tl];
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) a[u] = xrow[j[u]];
#pragma unroll
            for (int u = 0; u < 4; ++u) acc = mfma32(a[u], b[u], acc);
        }
        for (; p < pb; p += 2) {
            const int q = p + kh;
            float a = 0.0f, b = 0.0f;
            if (q < pb) {
                a = xrow[clampi(indices[q], 0, Kb - 1)];
                b = data[int64_t(q) * 32 + tl];
            }
            acc = mfma32(a, b, acc);
        }
    }
    __device__ static void store(const Acc &acc, float *__restrict__ Y, int64_t ldy, int64_t t0,
                                 int64_t T, int64_t n0, const float *__restrict__ bias) {
        const int lane = threadIdx.x & 63, tl = lane & 31, kh = lane >> 5;
        const float bv = bias ? bias[n0 + tl] : 0.0f;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int64_t t = t0 + 8 * (v >> 2) + 4 * kh + (v & 3);
            if (t < T) Y[t * ldy + n0 + tl] = acc[v] + bv;
        }
    }
};

// 16x1 blocks, v_mfma_f32_16x16x4_f32 on two 16-token halves.  acc[h][v] of lane l holds
// Y[t0 + 16h + 4*(l/16) + v][n0 + l%16].
template <>
struct Engine<16, 1> {
    struct Acc {
        floatx4 h[2];
    };
    static constexpr int kRegs = 8;
    static constexpr int kPad = 1;
    __device__ static void zero(Acc &a) {
#pragma unroll
        for (int v = 0; v < 4; ++v) a.h[0][v] = a.h[1][v] = 0.0f;
    }
    __device__ static void accumulate(Acc &acc, int pa, int pb, const int *__restrict__ indices,
                                      const float *__restrict__ data, const float *Xs, int XP,
                                      int Kb) {
        const int lane = threadIdx.x & 63, tl = lane & 15, kq = lane >> 4;
        const float *x0 = Xs + tl * XP;
        const float *x1 = Xs + (16 + tl) * XP;
        int p = pa;
        for (; p + 16 <= pb; p += 16) {
            int j[4];
            float b[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int q = p + 4 * u + kq;
                j[u] = clampi(indices[q], 0, Kb - 1);
                b[u] = data[int64_t(q) * 16 + tl];
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const float a0 = x0[j[u]], a1 = x1[j[u]];
                acc.h[0] = mfma16(a0, b[u], acc.h[0]);
                acc.h[1] = mfma16(a1, b[u], acc.h[1]);
            }
        }
        for (; p < pb; p += 4) {
            const int q = p + kq;
            float a0 = 0.0f, a1 = 0.0f, b = 0.0f;
            if (q < pb) {
                const int jj = clampi(indices[q], 0, Kb - 1);
                a0 = x0[jj];
                a1 = x1[jj];
                b = data[int64_t(q) * 16 + tl];
            }
            acc.h[0] = mfma16(a0, b, acc.h[0]);
            acc.h[1] = mfma16(a1, b, acc.h[1]);
        }
    }
    __device__ static void store(const Acc &acc, float *__restrict__ Y, int64_t ldy, int64_t t0,
                                 int64_t T, int64_t n0, const float *__restrict__ bias) {
        const int lane = threadIdx.x & 63, tl = lane & 15, kq = lane >> 4;
        const float bv = bias ? bias[n0 + tl] : 0.0f;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int64_t t = t0 + 16 * h + 4 * kq + v;
                if (t < T) Y[t * ldy + n0 + tl] = acc.h[h][v] + bv;
            }
        }
    }
};

// 32x32 blocks, v_mfma_f32_32x32x2_f32.  For block-column step u (8 columns) and e in 0..3,
// lane l's k-slot l/32 stands for c = 8u + 4*(l/32) + e in both operands.
template <>
struct Engine<32, 32> {
    using Acc = floatx16;
    static constexpr int kRegs = 16;
    static constexpr int kPad = 4;
    __device__ static void zero(Acc &a) { Engine<32, 1>::zero(a); }
    __device__ static void load_block(floatx4 (&d)[4], const float *__restrict__ data, int p,
                                      int tl, int kh) {
        const floatx4 *blk = reinterpret_cast<const floatx4 *>(data + int64_t(p) * 1024);
#pragma unroll
        for (int u = 0; u < 4; ++u) d[u] = blk[tl * 8 + 2 * u + kh];
    }
    __device__ static void accumulate(Acc &acc, int pa, int pb, const int *__restrict__ indices,
                                      const float *__restrict__ data, const float *Xs, int XP,
                                      int Kb) {
        const int lane = threadIdx.x & 63, tl = lane & 31, kh = lane >> 5;
        const float *xrow = Xs + tl * XP + 4 * kh;
        if (pa >= pb) return;
        floatx4 d[4], dn[4];
        int j = clampi(indices[pa], 0, Kb - 1);
        load_block(d, data, pa, tl, kh);
        for (int p = pa; p < pb; ++p) {
            int jn = j;
            if (p + 1 < pb) {
                jn = clampi(indices[p + 1], 0, Kb - 1);
                load_block(dn, data, p + 1, tl, kh);
            }
            const float *xb = xrow + j * 32;
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const floatx4 a = *reinterpret_cast<const floatx4 *>(xb + 8 * u);
#pragma unroll
                for (int e = 0; e < 4; ++e) acc = mfma32(a[e], d[u][e], acc);
            }
            if (p + 1 < pb) {
#pragma unroll
                for (int u = 0; u < 4; ++u) d[u] = dn[u];
            }
            j = jn;
        }
    }
    __device__ static void store(const Acc &acc, float *__restrict__ Y, int64_t ldy, int64_t t0,
                                 int64_t T, int64_t n0, const float *__restrict__ bias) {
        Engine<32, 1>::store(acc, Y, ldy, t0, T, n0, bias);
    }
};

// 16x16 blocks, v_mfma_f32_16x16x4_f32 on two 16-token halves.  Lane l loads row l%16,
// columns 4*(l/16)..+3 of the block (the whole block in one instruction); k-slot l/16 of step
// e stands for c = 4*(l/16) + e.
template <>
struct Engine<16, 16> {
    using Acc = Engine<16, 1>::Acc;
    static constexpr int kRegs = 8;
    static constexpr int kPad = 4;
    __device__ static void zero(Acc &a) { Engine<16, 1>::zero(a); }
    __device__ static void accumulate(Acc &acc, int pa, int pb, const int *__restrict__ indices,
                                      const float *__restrict__ data, const float *Xs, int XP,
                                      int Kb) {
        const int lane = threadIdx.x & 63, tl = lane & 15, kq = lane >> 4;
        const float *x0 = Xs + tl * XP + 4 * kq;
        const float *x1 = Xs + (16 + tl) * XP + 4 * kq;
        int p = pa;
        for (; p + 2 <= pb; p += 2) {
            int j[2];
            floatx4 d[2];
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                j[u] = clampi(indices[p + u], 0, Kb - 1);
                d[u] = reinterpret_cast<const floatx4 *>(data + int64_t(p + u) * 256)[tl * 4 + kq];
            }
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const floatx4 a0 = *reinterpret_cast<const floatx4 *>(x0 + j[u] * 16);
                const floatx4 a1 = *reinterpret_cast<const floatx4 *>(x1 + j[u] * 16);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    acc.h[0] = mfma16(a0[e], d[u][e], acc.h[0]);
                    acc.h[1] = mfma16(a1[e], d[u][e], acc.h[1]);
                }
            }
        }
        if (p < pb) {
            const int jj = clampi(indices[p], 0, Kb - 1);
            const floatx4 d = reinterpret_cast<const floatx4 *>(data + int64_t(p) * 256)[tl * 4 + kq];
            const floatx4 a0 = *reinterpret_cast<const floatx4 *>(x0 + jj * 16);
            const floatx4 a1 = *reinterpret_cast<const floatx4 *>(x1 + jj * 16);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                acc.h[0] = mfma16(a0[e], d[e], acc.h[0]);
                acc.h[1] = mfma16(a1[e], d[e], acc.h[1]);
            }
        }
    }
    __device__ static void store(const Acc &acc, float *__restrict__ Y, int64_t ldy, int64_t t0,
                                 int64_t T, int64_t n0, const float *__restrict__ bias) {
        Engine<16, 1>::store(acc, Y, ldy, t0, T, n0, bias);
    }
};

// Register v of an accumulator tile (the tile is a 16-wide vector or two 4-wide vectors).
__device__ __forceinline__ float acc_get(const floatx16 &a, int v) { return a[v]; }
__device__ __forceinline__ void acc_add(floatx16 &a, int v, float x) { a[v] += x; }
__device__ __forceinline__ float acc_get(const Engine<16, 1>::Acc &a, int v) {
    return a.h[v >> 2][v & 3];
}
__device__ __forceinline__ void acc_add(Engine<16, 1>::Acc &a, int v, float x) {
    a.h[v >> 2][v & 3] += x;
}

// -------------------------------------------------------------------------------- the kernel

template <int R, int C, int NW>
__global__ __launch_bounds__(NW * 64) void spmm_tiled_kernel(
    const float *__restrict__ X, int64_t T, int64_t ldx, int K, const int32_t *__restrict__ indptr,
    const int32_t *__restrict__ indices, const float *__restrict__ data, int nnzb, int Nb, int Kb,
    const float *__restrict__ bias, float *__restrict__ Y, int64_t ldy, int num_tiles,
    int slices, int XP, int indptr_words, int x_vec4) {
    using E = Engine<R, C>;
    extern __shared__ float smem[];
    int *s_indptr = reinterpret_cast<int *>(smem);
    float *Xs = smem + indptr_words;

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    constexpr int kThreads = NW * 64;

    // Workgroup -> (token tile, slice).  Workgroups are dealt to the 8 XCDs round robin, so
    // ids with equal (id mod 8) share an XCD; all slices of a tile get the same residue.
    const int g = blockIdx.x, xcd = g & 7, local = g >> 3;
    const int tile = (local / slices) * 8 + xcd, s = local % slices;
    if (tile >= num_tiles) return;
    const int64_t t0 = int64_t(tile) * kTT;

    for (int i = threadIdx.x; i <= Nb; i += kThreads) s_indptr[i] = clampi(indptr[i], 0, nnzb);

    // Stage X[t0 : t0 + 32][0 : K] into LDS (row pitch XP); rows past T are zero.
    if (x_vec4) {
        const int K4 = K >> 2;
        for (int f = threadIdx.x; f < kTT * K4; f += kThreads) {
            const int t = f / K4, c4 = f - t * K4;
            floatx4 v = {0.0f, 0.0f, 0.0f, 0.0f};
            if (t0 + t < T)
                v = *reinterpret_cast<const floatx4 *>(X + (t0 + t) * ldx + 4 * c4);
            float *dst = Xs + t * XP + 4 * c4;
            if constexpr (E::kPad == 4) {
                *reinterpret_cast<floatx4 *>(dst) = v;
            } else {
                dst[0] = v[0];
                dst[1] = v[1];
                dst[2] = v[2];
                dst[3] = v[3];
            }
        }
    } else {
        for (int f = threadIdx.x; f < kTT * K; f += kThreads) {
            const int t = f / K, c = f - t * K;
            Xs[t * XP + c] = (t0 + t < T) ? X[(t0 + t) * ldx + c] : 0.0f;
        }
    }
    __syncthreads();

    // This slice's block-rows and stored-block range.
    const int64_t k = s_indptr[Nb];
    const int row_lo = (s == 0) ? 0 : wave_lower_bound(s_indptr, Nb, int64_t(s) * k / slices);
    const int row_hi = (s == slices - 1)
                           ? Nb
                           : wave_lower_bound(s_indptr, Nb, int64_t(s + 1) * k / slices);
    const int64_t Q0 = s_indptr[row_lo], Q1 = s_indptr[row_hi];
    const int64_t span = Q1 > Q0 ? Q1 - Q0 : 0;
    auto wave_start = [&](int w) -> int64_t { return Q0 + span * w / NW; };
    const int64_t Pw = wave_start(wave), Pw1 = wave_start(wave + 1);

    // Rows owned by this wave: those whose first block lies in [Pw, Pw1) (last wave: all rows
    // up to the slice end, including trailing empty rows).
    int rlo = (wave == 0) ? row_lo : wave_lower_bound(s_indptr, Nb, Pw);
    rlo = rlo < row_lo ? row_lo : (rlo > row_hi ? row_hi : rlo);
    int rhi = (wave == NW - 1) ? row_hi : wave_lower_bound(s_indptr, Nb, Pw1);
    rhi = rhi < rlo ? rlo : (rhi > row_hi ? row_hi : rhi);

    // Head: blocks of [Pw, Pw1) that belong to the row started by an earlier wave.
    int64_t head_end = (rlo < rhi) ? int64_t(s_indptr[rlo]) : Pw1;
    head_end = head_end < Pw ? Pw : (head_end > Pw1 ? Pw1 : head_end);
    const bool has_head = head_end > Pw;
    typename E::Acc head;
    E::zero(head);
    if (has_head)
        E::accumulate(head, int(Pw), int(head_end), indices, data, Xs, XP, Kb);

    typename E::Acc acc;
    int tail_row = -1;
    for (int i = rlo; i < rhi; ++i) {
        const int pa = s_indptr[i];
        const int pe = s_indptr[i + 1];
        const int pb = pe < Pw1 ? pe : int(Pw1);
        E::zero(acc);
        E::accumulate(acc, pa, pb, indices, data, Xs, XP, Kb);
        if (pe > Pw1) {
            tail_row = i;
            break;
        }
        E::store(acc, Y, ldy, t0, T, int64_t(i) * R, bias);
    }

    // Combine rows cut by wave boundaries.  The X tile is dead now; reuse its LDS.
    __syncthreads();
    float *H = Xs;
    if (has_head) {
#pragma unroll
        for (int v = 0; v < E::kRegs; ++v)
            H[(wave * E::kRegs + v) * 64 + lane] = acc_get(head, v);
    }
    __syncthreads();
    if (tail_row >= 0) {
        // Every later wave whose range starts inside this row holds a head partial of it,
        // except waves with an empty range, which wrote nothing.
        const int64_t end = s_indptr[tail_row + 1];
        for (int w2 = wave + 1; w2 < NW && wave_start(w2) < end; ++w2) {
            if (wave_start(w2 + 1) == wave_start(w2)) continue;
#pragma unroll
            for (int v = 0; v < E::kRegs; ++v)
                acc_add(acc, v, H[(w2 * E::kRegs + v) * 64 + lane]);
        }
        E::store(acc, Y, ldy, t0, T, int64_t(tail_row) * R, bias);
    }
}

template <int R, int C, int NW>
bsr_status launch_variant(const TiledPlan &plan, const float *X, int64_t T, int64_t ldx,
                          const bsr_matrix_t *W, const float *bias, float *Y, int64_t ldy,
                          hipStream_t st) {
    const int K = int(W->n_cols), Nb = int(W->n_rows / R), Kb = int(W->n_cols / C);
    const int grid = ((plan.num_tiles + 7) / 8) * 8 * plan.slices;
    hipLaunchKernelGGL((spmm_tiled_kernel<R, C, NW>), dim3(grid), dim3(NW * 64), plan.lds_bytes,
                       st, X, T, ldx, K, W->indptr, W->indices,
                       static_cast<const float *>(W->data), int(W->nnzb), Nb, Kb, bias, Y, ldy,
                       plan.num_tiles, plan.slices, plan.x_pitch, plan.indptr_words,
                       plan.x_vec4);
    return launch_status();
}

}  // namespace

bool tiled_supported(int R, int C, int dtype) {
    if (dtype != BSR_F32) return false;
    return (R == 32 && C == 1) || (R == 16 && C == 1) || (R == 32 && C == 32) ||
           (R == 16 && C == 16);
}

int tiled_waves(int R, int C) { return (R == 32 && C == 32) ? 8 : 16; }

TiledPlan plan_tiled(const void *X, int64_t T, int64_t ldx, const bsr_matrix_t *W, int slices,
                     size_t lds_limit) {
    TiledPlan p{};
    const int R = W->R, C = W->C;
    if (!tiled_supported(R, C, W->dtype)) return p;
    const int64_t K = W->n_cols, Nb = W->n_rows / R;
    const int pad = (C == 1) ? 1 : 4;
    const int regs = (R == 32) ? 16 : 8;
    const int NW = tiled_waves(R, C);
    p.x_pitch = int(K + pad);
    p.indptr_words = int((Nb + 1 + 3) & ~int64_t(3));
    const size_t tile_bytes = size_t(kTT) * size_t(p.x_pitch) * 4;
    const size_t h_bytes = size_t(NW) * regs * 64 * 4;
    p.lds_bytes = size_t(p.indptr_words) * 4 + (tile_bytes > h_bytes ? tile_bytes : h_bytes);
    if (p.lds_bytes > lds_limit) return TiledPlan{};
    if (W->nnzb >= (int64_t(1) << 31) / (R * C)) return TiledPlan{};
    // Square kernels read 16-byte vectors from data; both kernels read X in float4 when the
    // rows allow it.
    const bool data_al = (reinterpret_cast<uintptr_t>(W->data) & 15) == 0;
    if (C > 1 && !data_al) return TiledPlan{};
    p.x_vec4 = ((reinterpret_cast<uintptr_t>(X) & 15) == 0 && K % 4 == 0 && ldx % 4 == 0) ? 1 : 0;
    p.num_tiles = int((T + kTT - 1) / kTT);
    p.slices = slices > 0 ? slices : 1;
    if (p.slices > Nb) p.slices = int(Nb);
    p.ok = true;
    return p;
}

bsr_status launch_spmm_tiled(const TiledPlan &plan, const void *X, int64_t T, int64_t ldx,
                             const bsr_matrix_t *W, const float *bias, float *Y, int64_t ldy,
                             void *stream) {
    hipStream_t st = as_stream(stream);
    const float *Xf = static_cast<const float *>(X);
    if (W->R == 32 && W->C == 1)
        return launch_variant<32, 1, 16>(plan, Xf, T, ldx, W, bias, Y, ldy, st);
    if (W->R == 16 && W->C == 1)
        return launch_variant<16, 1, 16>(plan, Xf, T, ldx, W, bias, Y, ldy, st);
    if (W->R == 32 && W->C == 32)
        return launch_variant<32, 32, 8>(plan, Xf, T, ldx, W, bias, Y, ldy, st);
    if (W->R == 16 && W->C == 16)
        return launch_variant<16, 16, 16>(plan, Xf, T, ldx, W, bias, Y, ldy, st);
    return BSR_ERR_UNSUPPORTED;
}

}  // namespace bsr
