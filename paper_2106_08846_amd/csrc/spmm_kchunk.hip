// BSR product on matrix cores for inputs too wide for one LDS X tile (in BERT-base, the
// 3072-column input of the feed-forward output layer: a 32-token fp32 tile of it would need
// 384 KB of LDS, and a workgroup has 160 KB):
//
//   Y[t][n] = bias[n] + sum over stored blocks p of block-row i = n / R of
//             sum over c < C of X[t][indices[p] * C + c] * data[p][n - iR][c]      (Sec. 2.2)
//
// The input columns are cut into chunks of chunk_blocks block-columns.  One workgroup covers 32
// tokens and one slice of block-rows; each wave owns up to kMR whole block-rows of the slice, or
// a slice of few rows gives each row a group of waves that split its blocks, and the waves keep
// their accumulators in registers from the first chunk to the last.  Per chunk:
//   * the workgroup stages X[t0 : t0 + 32][chunk columns] into LDS, in the layout the block
//     shape's unit reads (the same units and layouts as the tiled kernel);
//   * each wave finds where each of its rows leaves the chunk: indices ascend within a row, so
//     that is the first stored block whose column is past the chunk (one ballot per 64
//     indices), and runs the row's units from its current position up to there;
//   * the next chunk continues each row from where the previous one stopped, so every stored
//     block is visited once, in position order.
// A row tile starts at the bias and is stored once, after the last chunk (for a wave group,
// once the members' partial tiles have been added in member order).  The order of every sum is
// fixed by the plan, so results are bitwise reproducible.
#include <type_traits>

#include "device_common.h"
#include "spmm_tiled.h"
#include "spmm_units.h"

namespace bsr {

namespace {

constexpr int kNW = 16;     // waves per workgroup
constexpr int kMR = 2;      // block-rows per wave at most
constexpr int kGroups = 8;  // 64-word groups of an X row in flight per lane while staging

// A unit's column indices made relative to the chunk's first block-column.
template <typename Ops>
__device__ __forceinline__ void shift_cols(Ops &ops, int jlo) {
    if constexpr (std::is_array_v<decltype(ops.j)>) {
#pragma unroll
        for (int m = 0; m < int(std::extent_v<decltype(ops.j)>); ++m) ops.j[m] -= jlo;
    } else {
        ops.j -= jlo;
    }
}

template <int R, int C, bool BF, int W = 1>
__global__ __launch_bounds__(kNW * 64) void spmm_kchunk_kernel(const KchunkBatch batch) {
    using U = typename UnitOf<R, C, BF, W>::type;
    extern __shared__ float smem[];
    constexpr int kThreads = kNW * 64;
    const int lane = threadIdx.x & 63, wave = uniform(threadIdx.x >> 6);

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

    // Workgroup -> (token tile, slice), dealt to the 8 XCDs in contiguous ranges as in the
    // tiled kernel, so that the slices of a token tile share an L2.
    const int g = blockIdx.x, xcd = g & 7, rank = g >> 3;
    const int pairs = num_tiles * slices, per_xcd = (pairs + 7) >> 3;
    const int q = xcd * per_xcd + rank;
    if (rank >= per_xcd || q >= pairs) return;
    const int tile = q / slices, s = q - tile * slices;
    const int64_t t0 = int64_t(tile) * kTT;
    const int rows = int(T - t0 < kTT ? T - t0 : kTT);
    // Slice s holds block-rows [row_lo, row_hi): equal counts (the plan keeps <= kNW * kMR).
    const int row_lo = int(int64_t(s) * Nb / slices);
    const int row_hi = int(int64_t(s + 1) * Nb / slices);

    // LDS: the slice's bias, then the X chunk tile, then (transposed bf16 32x1) 2 KB of block
    // scratch per wave.
    float *s_bias = smem;
    float *Xs = smem + I.bias_words;
    char *wslot = reinterpret_cast<char *>(Xs) + I.wbuf_offset + wave * 2048;
    for (int i = threadIdx.x; i < (row_hi - row_lo) * R; i += kThreads)
        s_bias[i] = bias ? bias[int64_t(row_lo) * R + i] : 0.0f;

    // Rows of the waves.  A slice of at most kNW / 2 rows gives each row a group of G >= 2
    // waves (wave w: row w / G, member w % G), which split the row's blocks of every chunk into
    // G contiguous parts and add their partial tiles in member order at the end; otherwise
    // (G = 1) wave w owns rows row_lo + w + kNW * i, i < kMR.  Slot i of a wave holds row
    // row_of(i), or a row >= row_hi when the slot is unused.
    const int nr = row_hi - row_lo;
    const int G = 2 * nr <= kNW ? kNW / nr : 1;
    const int member = wave % G;
    auto row_of = [&](int i) -> int {
        if (G > 1) return (i == 0 && wave / G < nr) ? row_lo + wave / G : row_hi;
        return row_lo + wave + kNW * i;
    };
    int pos[kMR], end[kMR];
#pragma unroll
    for (int i = 0; i < kMR; ++i) {
        const int row = row_of(i);
        pos[i] = end[i] = 0;
        if (row < row_hi) {
            pos[i] = uniform(clampi(indptr[row], 0, nnzb));
            end[i] = uniform(clampi(indptr[row + 1], pos[i], nnzb));
        }
    }

    // Stage X[t0 : t0 + 32][jlo*C : jlo*C + cols] (rows past T and columns past the chunk read
    // 0 through the buffer ranges).  fp32 and widened bf16 tiles: row-major, pitch XP floats;
    // bf16 square tiles: row-major, pitch XP bf16, two columns per word; the transposed bf16
    // tile: column-major, 32 tokens per column at pitch XP bf16.  The R x 1 layouts get a zero
    // column at index cols, which masked lanes read.
    constexpr int kXBytes = BF ? 2 : 4;
    constexpr int kColsPerWord = U::kTileBF16 && !U::kTransposed ? 2 : 1;
    constexpr int kRowsPerWave = kTT / kNW;
    static_assert(kTT % kNW == 0, "every wave stages the same number of rows");
    auto stage = [&](int jlo, int cols) {
        const int words = (cols + kColsPerWord - 1) / kColsPerWord;
        __amdgpu_buffer_rsrc_t rx[kRowsPerWave];
#pragma unroll
        for (int r = 0; r < kRowsPerWave; ++r) {
            const int t = wave + kNW * r;
            const int tr = t < rows ? t : rows - 1;
            rx[r] = buffer_rsrc(static_cast<const char *>(X) +
                                    ((t0 + tr) * ldx + int64_t(jlo) * C) * kXBytes,
                                t < rows ? unsigned(cols) * kXBytes : 0u);
        }
        for (int w0 = 0; w0 < words; w0 += 64 * kGroups) {
            unsigned v[kRowsPerWave][kGroups];
#pragma unroll
            for (int r = 0; r < kRowsPerWave; ++r)
#pragma unroll
                for (int m = 0; m < kGroups; ++m) {
                    const int w = w0 + 64 * m + lane;
                    if constexpr (BF && (U::kTransposed || !U::kTileBF16))
                        v[r][m] = __builtin_amdgcn_raw_buffer_load_b16(rx[r], w * 2, 0, 0);
                    else
                        v[r][m] = __builtin_amdgcn_raw_buffer_load_b32(rx[r], w * 4, 0, 0);
                }
#pragma unroll
            for (int r = 0; r < kRowsPerWave; ++r) {
                const int t = wave + kNW * r;
#pragma unroll
                for (int m = 0; m < kGroups; ++m) {
                    const int w = w0 + 64 * m + lane;
                    if (w < words) {
                        if constexpr (U::kTransposed) {
                            reinterpret_cast<bf16_t *>(Xs)[w * XP + t] = bf16_t(v[r][m]);
                        } else {
                            unsigned x = v[r][m];
                            if constexpr (BF && !U::kTileBF16) x <<= 16;   // bf16 -> fp32, exact
                            reinterpret_cast<unsigned *>(Xs)[t * (XP / kColsPerWord) + w] = x;
                        }
                    }
                }
            }
        }
        if constexpr (U::kTransposed) {
            if (threadIdx.x < kTT) reinterpret_cast<bf16_t *>(Xs)[cols * XP + threadIdx.x] = 0;
        } else if constexpr (U::kPad == 1) {
            if (threadIdx.x < kTT) Xs[threadIdx.x * XP + cols] = 0.0f;
        }
    };

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

    // The units of positions [q0, qe) of one row against the chunk tile (kbw block-columns
    // from jlo), one unit's loads ahead; a partial last unit is masked.
    auto run = [&](typename U::Acc &a, int q0, int qe, int jlo, int kbw) {
        if (q0 >= qe) return;
        typename U::Ops A, B;
        U::load(A, q0, nnzb, indices, data);
        int qq = q0;
        while (true) {
            const int qn = qq + U::KB;
            const bool more = qn < qe;
            if (more) U::load(B, qn, nnzb, indices, data);
            shift_cols(A, jlo);
            if (qe - qq < U::KB) U::mask(A, qe - qq);
            U::mma(a, A, Xs, XP, kbw, wslot);
            if (!more) break;
            A = B;
            qq = qn;
        }
    };

    typename U::Acc acc[kMR];
    for (int c = 0; c < nchunks; ++c) {
        const int jlo = c * kcb;
        const int jhi = c + 1 == nchunks ? Kb : jlo + kcb;
        if (c > 0) __syncthreads();   // every wave is done with the previous chunk's tile
        stage(jlo, (jhi - jlo) * C);
        int cend[kMR];
#pragma unroll
        for (int i = 0; i < kMR; ++i)
            cend[i] = c + 1 == nchunks ? end[i] : crossing(pos[i], end[i], jhi);
        __syncthreads();
        if (c == 0) {
#pragma unroll
            for (int i = 0; i < kMR; ++i) {
                const int row = row_of(i);
                if (row < row_hi && member == 0) U::init(acc[i], s_bias, (row - row_lo) * R);
                else U::zero(acc[i]);
            }
        }
#pragma unroll
        for (int i = 0; i < kMR; ++i) {
            // This member's part of the row's positions in the chunk (all of them when G = 1).
            const int len = cend[i] - pos[i];
            const int lo = pos[i] + int((int64_t(len) * member) / G);
            const int hi = pos[i] + int((int64_t(len) * (member + 1)) / G);
            run(acc[i], lo, hi, jlo, jhi - jlo);
            pos[i] = cend[i];
        }
    }

    TileOut out;
    out.ldy4 = int(ldy) * 4;
    out.rsrc = buffer_rsrc(Y + t0 * ldy, unsigned(rows) * unsigned(out.ldy4));
    if (G == 1) {
#pragma unroll
        for (int i = 0; i < kMR; ++i) {
            const int row = row_of(i);
            if (row < row_hi) U::store(acc[i], out, row * R);
        }
        return;
    }
    // Wave groups: members 1 .. G-1 leave their partial tiles in LDS (the X tile is dead after
    // the barrier); member 0 adds them in member order and stores the row.
    constexpr int kSlot = U::kRegs * 64;
    float *P = Xs;
    __syncthreads();
    if (member > 0) {
#pragma unroll
        for (int v = 0; v < U::kRegs; ++v) P[(wave * U::kRegs + v) * 64 + lane] = U::get(acc[0], v);
    }
    __syncthreads();
    const int row = row_of(0);
    if (member == 0 && row < row_hi) {
        for (int m = 1; m < G; ++m) {
            const float *src = P + (wave + m) * kSlot;
#pragma unroll
            for (int v = 0; v < U::kRegs; ++v) U::add(acc[0], v, src[v * 64 + lane]);
        }
        U::store(acc[0], out, row * R);
    }
}

template <int R, int C, bool BF, int W = 1>
bsr_status launch_kchunk_variant(const KchunkBatch &batch, dim3 grid, size_t lds, hipStream_t st,
                                 const LaunchEvents &ev) {
    launch_kernel(spmm_kchunk_kernel<R, C, BF, W>, grid, dim3(kNW * 64), lds, st, ev, batch);
    return launch_status();
}

}  // namespace

KchunkPlan plan_kchunk(const void *X, int64_t T, int64_t ldx, const bsr_matrix_t *W,
                       int64_t ldy, int slices, size_t lds_limit) {
    KchunkPlan kp{};
    const int R = W->R, C = W->C;
    if (!tiled_supported(R, C, W->dtype)) return kp;
    const int64_t K = W->n_cols, Nb = W->n_rows / R, Kb = K / C;
    const bool bf = W->dtype == BSR_BF16;
    const bool transposed = bf && R == 32 && C == 1;        // Unit<32, 1, true>::kTransposed
    const bool tile_bf16 = bf && (C > 1 || transposed);     // Unit<R, C, BF>::kTileBF16
    // Widest pitch padding tile_pitch() adds (the chunk width is not known yet).
    const int pad = (C == 1) ? (R == 16 ? 32 : 2) : 8;
    // Slices: at least enough that no wave owns more than kMR rows, at most one row each.
    int64_t S = slices > 0 ? slices : 1;
    const int64_t min_s = (Nb + kNW * kMR - 1) / (kNW * kMR);
    if (S < min_s) S = min_s;
    if (S > Nb) S = Nb;
    const int64_t slice_rows = (Nb + S - 1) / S;
    TiledPlan &p = kp.base;
    p.bias_words = int((slice_rows * R + 3) & ~int64_t(3));
    // The widest chunk (input columns) whose tile fits beside the bias.
    const int64_t avail = int64_t(lds_limit) - int64_t(p.bias_words) * 4;
    int64_t cmax;
    if (transposed) cmax = (avail - kNW * 2048 - 255) / 72 - 1;
    else if (tile_bf16) cmax = avail / (kTT * 2) - pad;
    else cmax = avail / (kTT * 4) - pad;
    const int64_t kcb_max = cmax / C;
    if (kcb_max < 1) return KchunkPlan{};
    // Equal chunks, as few as fit.
    const int64_t nch = (Kb + kcb_max - 1) / kcb_max;
    const int64_t kcb = (Kb + nch - 1) / nch;
    const int64_t kc = kcb * C;
    size_t tile_bytes;
    if (transposed) {
        p.x_pitch = 36;
        p.wbuf_offset = int(((kc + 1) * 72 + 255) & ~int64_t(255));
        tile_bytes = size_t(p.wbuf_offset) + size_t(kNW) * 2048;
    } else {
        p.x_pitch = int(tile_pitch(R, C, tile_bf16, kc));
        p.wbuf_offset = 0;
        tile_bytes = size_t(kTT) * size_t(p.x_pitch) * (tile_bf16 ? 2 : 4);
    }
    // After the last chunk the tile's LDS holds the partial tiles of wave groups.
    const size_t partial_bytes = size_t(kNW) * (R == 32 ? 16 : 8) * 64 * 4;
    if (tile_bytes < partial_bytes) tile_bytes = partial_bytes;
    p.lds_bytes = size_t(p.bias_words) * 4 + tile_bytes;
    if (p.lds_bytes > lds_limit) return KchunkPlan{};
    // Buffer ranges are 32-bit (block data, one X row, a 32-row tile of Y); square units read
    // 16-byte vectors of data; bf16 square tiles load X in dwords.
    if (W->nnzb * R * C >= (int64_t(1) << 29)) return KchunkPlan{};
    if (ldy >= (int64_t(1) << 24) || K >= (int64_t(1) << 24)) return KchunkPlan{};
    if (C > 1 && (reinterpret_cast<uintptr_t>(W->data) & 15) != 0) return KchunkPlan{};
    if (bf && C > 1 && ((reinterpret_cast<uintptr_t>(X) & 3) != 0 || (ldx & 1) != 0))
        return KchunkPlan{};
    p.num_tiles = int((T + kTT - 1) / kTT);
    p.slices = int(S);
    p.ok = true;
    kp.chunk_blocks = int(kcb);
    kp.nchunks = int(nch);
    return kp;
}

bsr_status launch_spmm_kchunk(const KchunkWork *work, int n, void *stream,
                              const LaunchEvents &ev) {
    if (n < 1 || n > kMaxItems) return BSR_ERR_ARG;
    const int R = work[0].W->R, C = work[0].W->C;
    KchunkBatch batch{};
    batch.n = n;
    int gx = 0;
    size_t lds = 0;
    for (int i = 0; i < n; ++i) {
        const KchunkWork &w = work[i];
        if (w.W->R != R || w.W->C != C || w.W->dtype != work[0].W->dtype) return BSR_ERR_ARG;
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
        it.bias_words = w.plan.base.bias_words;
        it.wbuf_offset = w.plan.base.wbuf_offset;
        it.chunk_blocks = w.plan.chunk_blocks;
        it.nchunks = w.plan.nchunks;
        const int wgs = ((w.plan.base.num_tiles * w.plan.base.slices + 7) / 8) * 8;
        if (wgs > gx) gx = wgs;
        if (w.plan.base.lds_bytes > lds) lds = w.plan.base.lds_bytes;
    }
    const dim3 grid(gx, n);
    hipStream_t st = as_stream(stream);
    int64_t blocks = 0, rows = 0;
    for (int i = 0; i < n; ++i) {
        blocks += work[i].W->nnzb;
        rows += work[i].W->n_rows / R;
    }
    if (R == 16 && C == 16 && blocks >= kWideUnitRowBlocks * rows) {
        if (work[0].W->dtype == BSR_BF16)
            return launch_kchunk_variant<16, 16, true, 4>(batch, grid, lds, st, ev);
        return launch_kchunk_variant<16, 16, false, 4>(batch, grid, lds, st, ev);
    }
    if (work[0].W->dtype == BSR_BF16) {
        if (R == 32 && C == 1) return launch_kchunk_variant<32, 1, true>(batch, grid, lds, st, ev);
        if (R == 16 && C == 1) return launch_kchunk_variant<16, 1, true>(batch, grid, lds, st, ev);
        if (R == 32 && C == 32) return launch_kchunk_variant<32, 32, true>(batch, grid, lds, st, ev);
        if (R == 16 && C == 16) return launch_kchunk_variant<16, 16, true>(batch, grid, lds, st, ev);
    } else {
        if (R == 32 && C == 1) return launch_kchunk_variant<32, 1, false>(batch, grid, lds, st, ev);
        if (R == 16 && C == 1) return launch_kchunk_variant<16, 1, false>(batch, grid, lds, st, ev);
        if (R == 32 && C == 32) return launch_kchunk_variant<32, 32, false>(batch, grid, lds, st, ev);
        if (R == 16 && C == 16) return launch_kchunk_variant<16, 16, false>(batch, grid, lds, st, ev);
    }
    return BSR_ERR_UNSUPPORTED;
}

}  // namespace bsr
