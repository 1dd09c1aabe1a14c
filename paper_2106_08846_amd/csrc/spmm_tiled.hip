// Tiled BSR product on gfx950 matrix cores (fp32 or bf16 inputs, fp32 accumulate).
//
// Y[t][n] = bias[n] + sum over stored blocks p of block-row i = n / R of
//           sum over c < C of X[t][indices[p] * C + c] * data[p][n - iR][c]          (Sec. 2.2)
//
// For one block-row and a tile of tokens this is a small dense product once the input columns
// named by `indices` are gathered: Y_tile (tokens x R) += X_tile[:, cols] (tokens x m*C) times
// the row's blocks (m*C x R).  The matrix-core units of spmm_units.h run it on MFMA.
//
// Work decomposition (one workgroup = 32 tokens x one slice of block-rows):
//   * the X tile [32 tokens][K] is staged once into LDS: coalesced buffer loads of one word per
//     lane (constant offsets in the instruction) and conflict-free LDS stores, with row pitch
//     K+1 (R x 1: conflict-free 4-byte gathers of one column for 32 tokens), K+4 or K+8
//     (square blocks, fp32 or bf16: 16-byte aligned rows), or transposed with a 72-byte column
//     pitch (bf16 32x1, for the LDS transpose reads); the bias is staged beside it and is the
//     initial value of every row the workgroup finishes;
//   * slices hold whole block-rows, balanced by stored-block count;
//   * inside a slice the stored blocks are split evenly over the waves (so skewed rows are
//     spread over several waves); a block-row cut by a wave boundary is summed by the wave where
//     it starts, adding the other waves' partial tiles from LDS in wave order after a barrier.
//     The summation order is fixed by the launch shape, so results are bitwise reproducible.
//   * workgroup ids are mapped so that the slices of one token tile run on the same XCD and
//     share its L2 for the X tile.
#include <type_traits>

#include "device_common.h"
#include "spmm_tiled.h"
#include "spmm_units.h"

namespace bsr {

namespace {

// -------------------------------------------------------------------------------- the kernel

template <int R, int C, int NW, bool BF, int W = 1>
__global__ __launch_bounds__(NW * 64) void spmm_tiled_kernel(const TiledBatch batch) {
    using U = typename UnitOf<R, C, BF, W>::type;
    extern __shared__ float smem[];

    // The wave index is uniform across a wave; readfirstlane tells the compiler so, which
    // keeps all loop and row bookkeeping in scalar registers with scalar branches.
    const int lane = threadIdx.x & 63, wave = uniform(threadIdx.x >> 6);
    constexpr int kThreads = NW * 64;

    // This workgroup's product is blockIdx.y, so its descriptor's address is known without a
    // lookup and every field arrives in one round of scalar loads.
    const int g = blockIdx.x;
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
    // LDS: indptr, bias (N floats), then the X tile (fp32, or bf16 for the bf16 square units;
    // reused for partial tiles at the end).
    int *s_indptr = reinterpret_cast<int *>(smem);
    float *s_bias = smem + I.indptr_words;
    float *Xs = s_bias + I.bias_words;

    // The descriptor's fields are pinned here, ahead of the early exit below; otherwise the
    // compiler sinks their loads past it and the X-tile loads wait for a second round.
    asm volatile("" ::"s"(X), "s"(T), "s"(ldx), "s"(ldy), "s"(indptr), "s"(indices), "s"(data),
                 "s"(bias), "s"(Y));
    asm volatile("" ::"s"(K), "s"(nnzb), "s"(Nb), "s"(Kb), "s"(num_tiles), "s"(slices), "s"(XP),
                 "s"(I.indptr_words), "s"(I.bias_words), "s"(I.wbuf_offset));

    // Workgroup -> (token tile, slice).  Workgroups are dealt to the 8 XCDs round robin in
    // dispatch order (x fastest, and the grid's x extent is a multiple of 8), so ids with equal
    // blockIdx.x mod 8 share an XCD.  The item's (tile, slice) pairs, in tile-major order, are
    // cut into 8 contiguous ranges, one per XCD: every XCD gets work, and the slices of a tile
    // stay on as few XCDs (L2s) as possible.
    const int xcd = g & 7, rank = g >> 3;
    const int pairs = num_tiles * slices, per_xcd = (pairs + 7) >> 3;
    const int q = xcd * per_xcd + rank;
    if (rank >= per_xcd || q >= pairs) return;
    const int tile = q / slices, s = q - tile * slices;
    const int64_t t0 = int64_t(tile) * kTT;

    // Stage X[t0 : t0 + 32][0 : K] into LDS (row pitch XP elements).  Each wave moves whole
    // rows: per 64 lanes one coalesced buffer load (constant offsets go in the instruction) and
    // one conflict-free LDS store of consecutive words.  A row's loads are all issued before
    // its stores.  fp32 X and the widened bf16 X move one column per lane; a bf16 tile moves
    // two columns (one dword) per lane.  Rows past T are zero, and so is the pad column K of
    // the R x 1 layout.
    const int rows = int(T - t0 < kTT ? T - t0 : kTT);
    constexpr int kXBytes = BF ? 2 : 4;
    constexpr int kColsPerLane = U::kTileBF16 && !U::kTransposed ? 2 : 1;
    constexpr int kRowsPerWave = kTT / NW;
    static_assert(kTT % NW == 0, "every wave stages the same number of rows");

    // The prologue overlaps the latencies of indptr, the X tile and the first unit:
    //   (1) every wave loads indptr into registers, the bias, and then its X-tile rows;
    //   (2) as soon as indptr arrives, the wave computes its share of the slice from registers
    //       (ballots and lane reads; no LDS, no barrier) and issues its first unit's loads;
    //   (3) indptr, bias and the X tile are written to LDS and one barrier ends the prologue.
    // A product with 256 or more block-rows copies indptr to LDS first and searches it there.
    constexpr int kIpChunks = 4;   // indptr entries per wave in registers: 64 per chunk
    constexpr int kBiasPer = 4;    // bias entries per thread staged through registers
    const bool reg_part = Nb < 64 * kIpChunks;
    int ip[kIpChunks];   // indptr[64 j + lane]
    float bv[kBiasPer];
    {
        const __amdgpu_buffer_rsrc_t rip = buffer_rsrc(indptr, unsigned(Nb + 1) * 4u);
        const __amdgpu_buffer_rsrc_t rb = buffer_rsrc(bias, bias ? unsigned(Nb * R) * 4u : 0u);
        // Large products skip these loads: an offset past the range reads 0 without a fetch.
        const unsigned off = reg_part ? unsigned(lane) * 4u : 0x7ffff000u;
#pragma unroll
        for (int j = 0; j < kIpChunks; ++j)
            ip[j] = __builtin_amdgcn_raw_buffer_load_b32(rip, off + 256 * j, 0, 0);
#pragma unroll
        for (int u = 0; u < kBiasPer; ++u)
            bv[u] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                                  rb, (threadIdx.x + u * kThreads) * 4, 0, 0));
    }

    // X tile staging, split into loads (into v) and LDS stores so that other work fits in
    // between.  Row-major layout (pitch XP elements): per 64 lanes one coalesced load of one
    // 32-bit word (fp32, widened bf16, or a pair of bf16 columns) and one conflict-free LDS
    // store.  Transposed layout (bf16 32x1): one bf16 per lane, stored to column c at token t.
    const int lane_words = (K + kColsPerLane - 1) / kColsPerLane;   // LDS words per row
    unsigned v[kRowsPerWave][kStageChunks];
    auto x_load = [&](int c0) {
#pragma unroll
        for (int r = 0; r < kRowsPerWave; ++r) {
            const int t = wave + NW * r;
            // Rows past T get an empty range (every load returns 0); the base is any valid row.
            const int tr = t < rows ? t : rows - 1;
            const __amdgpu_buffer_rsrc_t rx =
                buffer_rsrc(static_cast<const char *>(X) + (t0 + tr) * ldx * kXBytes,
                            t < rows ? unsigned(K) * kXBytes : 0u);
#pragma unroll
            for (int m = 0; m < kStageChunks; ++m) {
                // No guard needed: each row's buffer range ends at column K, so lanes past it
                // read 0.
                if constexpr (BF && (U::kTransposed || !U::kTileBF16))
                    v[r][m] = __builtin_amdgcn_raw_buffer_load_b16(rx, (c0 + lane) * 2 + 128 * m,
                                                                   0, 0);
                else
                    v[r][m] = __builtin_amdgcn_raw_buffer_load_b32(rx, (c0 + lane) * 4 + 256 * m,
                                                                   0, 0);
            }
        }
    };
    // Branch-free stores (straight-line code keeps the prologue short to fetch: every launch
    // starts with a cold instruction cache).  With `clamp`, a lane past the end of the row
    // (it loaded 0: the row's buffer range ends there) stores to the first word after the
    // row, which is padding that holds 0 anyway; without, every column of the group exists.
    auto x_store = [&](int c0, auto clamp) {
#pragma unroll
        for (int r = 0; r < kRowsPerWave; ++r) {
            const int t = wave + NW * r;
            if constexpr (U::kTransposed) {
                bf16_t *xt = reinterpret_cast<bf16_t *>(Xs) + t;
#pragma unroll
                for (int m = 0; m < kStageChunks; ++m) {
                    const int c = c0 + 64 * m + lane;
                    xt[(decltype(clamp)::value ? min(c, K) : c) * XP] = bf16_t(v[r][m]);
                }
            } else {
                // Row t of the tile as 32-bit words (fp32 columns, or pairs of bf16 columns).
                unsigned *dst = reinterpret_cast<unsigned *>(Xs) + t * (XP / kColsPerLane);
#pragma unroll
                for (int m = 0; m < kStageChunks; ++m) {
                    unsigned w = v[r][m];
                    if constexpr (BF && !U::kTileBF16) w <<= 16;   // bf16 -> fp32, exact
                    const int c = c0 + 64 * m + lane;
                    dst[decltype(clamp)::value ? min(c, lane_words) : c] = w;
                }
            }
        }
    };
    using Clamp = std::true_type;
    using NoClamp = std::false_type;
    x_load(0);

    // The wave's share of the slice.  Slices hold whole block-rows, balanced by stored-block
    // count: slice s covers rows [row_lo, row_hi) where row_lo is the first row whose start
    // is >= floor(s k / slices).  The slice's blocks [Q0, Q1) are split evenly over the waves
    // (wave w: [Pw, Pw1)).  A wave owns the rows whose first block lies in its range (the last
    // wave also owns trailing empty rows); blocks at the front of its range that belong to
    // row rlo - 1 are a head, summed into that row by the wave that owns it.
    int64_t k, Q0, Q1;
    int row_lo, row_hi, Pw, Pw1, rlo, rhi, head_end, row, p, end;
    // Wave starts, one per lane: ws = start of wave `lane`, wsn = start of wave lane + 1.
    int ws = 0, wsn = 0;
    auto share = [&](auto lower_bound) {
        // floor(span l / NW) in 32-bit parts (span < 2^29, l <= 64).
        static_assert(NW == 16, "wave starts use a division by 16");
        const unsigned span = unsigned(Q1 - Q0), hi = span >> 4, lo = span & 15u;
        const unsigned l0 = unsigned(lane), l1 = l0 + 1;
        ws = int(Q0) + int(hi * l0 + ((lo * l0) >> 4));
        wsn = int(Q0) + int(hi * l1 + ((lo * l1) >> 4));
        Pw = __builtin_amdgcn_readlane(ws, wave);
        Pw1 = __builtin_amdgcn_readlane(wsn, wave);
        rlo = (wave == 0) ? row_lo : lower_bound(int64_t(Pw));
        rlo = rlo < row_lo ? row_lo : (rlo > row_hi ? row_hi : rlo);
        rhi = (wave == NW - 1) ? row_hi : lower_bound(int64_t(Pw1));
        rhi = rhi < rlo ? rlo : (rhi > row_hi ? row_hi : rhi);
    };
    // The register partition, over the first NCH chunks of indptr (a product with fewer than
    // 64 block-rows runs the one-chunk instance: less code to fetch on the way to its first
    // unit).
    auto reg_partition = [&](auto nch) {
        constexpr int NCH = decltype(nch)::value;
#pragma unroll
        for (int j = 0; j < NCH; ++j) ip[j] = clampi(ip[j], 0, nnzb);
        // Entry i (uniform, <= Nb) of a register-resident array: one lane read per chunk and a
        // scalar select (a dynamic register index would send the array to scratch memory).
        auto lane_read = [&](const int(&a)[kIpChunks], int i) -> int {
            const int l = i & 63, c = i >> 6;
            int v = __builtin_amdgcn_readlane(a[0], l);
#pragma unroll
            for (int j = 1; j < NCH; ++j) {
                const int x = __builtin_amdgcn_readlane(a[j], l);
                v = c == j ? x : v;
            }
            return v;
        };
        // Number of rows i < Nb meeting a per-entry predicate; for a monotone predicate on
        // the non-decreasing indptr this is a lower bound.  (Lane masks of the rows < Nb are
        // formed once; each count is then one compare, mask and bit count per chunk.)
        unsigned long long in_rows[NCH];
#pragma unroll
        for (int j = 0; j < NCH; ++j) in_rows[j] = __ballot(64 * j + lane < Nb);
        auto count_rows = [&](auto pred) -> int {
            int c = 0;
#pragma unroll
            for (int j = 0; j < NCH; ++j) c += __popcll(__ballot(pred(ip[j])) & in_rows[j]);
            return c;
        };
        k = lane_read(ip, Nb);
        // indptr[i] < floor(s k / slices)  <=>  (indptr[i] + 1) slices <= s k.
        auto slice_start = [&](int s2) -> int {
            const uint64_t sk = uint64_t(s2) * uint64_t(k);
            return count_rows([&](int x) { return uint64_t(x + 1) * uint64_t(slices) <= sk; });
        };
        row_lo = (s == 0) ? 0 : slice_start(s);
        row_hi = (s == slices - 1) ? Nb : slice_start(s + 1);
        Q0 = lane_read(ip, row_lo);
        Q1 = lane_read(ip, row_hi);
        if (Q1 < Q0) Q1 = Q0;
        share([&](int64_t v) { return count_rows([&](int x) { return x < int(v); }); });
        head_end = (rlo < rhi) ? lane_read(ip, rlo) : Pw1;
        head_end = head_end < Pw ? Pw : (head_end > Pw1 ? Pw1 : head_end);
        if (head_end > Pw) {
            row = rlo - 1;
            p = Pw;
            end = head_end;
        } else {
            // First owned row with blocks.  Rows rlo, rlo + 1, ... that start where rlo starts
            // are empty except the last of them, which is the last row i with indptr[i] <= v
            // (a prefix of the non-decreasing indptr); it has blocks if its end exceeds v.
            row = rhi;
            p = end = 0;
            if (rlo < rhi) {
                const int v = lane_read(ip, rlo);
                const int c = count_rows([&](int x) { return x < v + 1; });
                const int e = lane_read(ip, c);
                if (c - 1 >= rlo && c - 1 < rhi && e > v) {
                    row = c - 1;
                    p = v;
                    end = e < Pw1 ? e : Pw1;
                }
            }
        }
    };
    if (__builtin_expect(Nb < 64, 1)) {
        reg_partition(std::integral_constant<int, 1>{});
    } else if (__builtin_expect(reg_part, 1)) {
        reg_partition(std::integral_constant<int, kIpChunks>{});
    } else {
        for (int i = threadIdx.x; i <= Nb; i += kThreads) s_indptr[i] = clampi(indptr[i], 0, nnzb);
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
        k = uniform(s_indptr[Nb]);
        row_lo = (s == 0) ? 0 : uniform(wave_lower_bound(s_indptr, Nb, int64_t(s) * k / slices));
        row_hi = (s == slices - 1)
                     ? Nb
                     : uniform(wave_lower_bound(s_indptr, Nb, int64_t(s + 1) * k / slices));
        Q0 = uniform(s_indptr[row_lo]);
        Q1 = uniform(s_indptr[row_hi]);
        if (Q1 < Q0) Q1 = Q0;
        share([&](int64_t v) { return uniform(wave_lower_bound(s_indptr, Nb, v)); });
        head_end = (rlo < rhi) ? uniform(s_indptr[rlo]) : Pw1;
        head_end = head_end < Pw ? Pw : (head_end > Pw1 ? Pw1 : head_end);
        row = rlo - 1;
        p = Pw;
        end = head_end;
        if (head_end <= Pw) {
            for (row = rlo; row < rhi; ++row) {
                p = uniform(s_indptr[row]);
                const int e = uniform(s_indptr[row + 1]);
                if (p < e) {
                    end = e < Pw1 ? e : Pw1;
                    break;
                }
            }
            if (row >= rhi) p = end = 0;
        }
    }
    const bool has_head = head_end > Pw;

    // First row after r with blocks (rhi if none); returns its start and clipped end.  Reads
    // the LDS copy of indptr (complete after the prologue's barrier).
    auto next_row = [&](int r, int &start, int &end_) -> int {
        for (++r; r < rhi; ++r) {
            start = uniform(s_indptr[r]);
            const int e = uniform(s_indptr[r + 1]);
            if (start < e) {
                end_ = e < Pw1 ? e : Pw1;
                return r;
            }
        }
        start = end_ = 0;
        return rhi;
    };
    // The first unit's loads (in flight during the tile stores).  Issued on every path, also
    // for a wave without blocks (an in-range position, never used), so the compiler can count
    // exactly which loads the tile stores below have to wait for.
    typename U::Ops A, B;
    U::load(A, row < rhi ? p : 0, nnzb, indices, data);

    // indptr (register path: wave 0) and bias into LDS.  Unconditional stores (threads past
    // the arrays write a spare word at the end of the indptr region), so that no load above is
    // sunk below the tile's loads.
    int *s_spare = s_indptr + I.indptr_words - 1;
    if (reg_part && wave == 0) {
#pragma unroll
        for (int j = 0; j < kIpChunks; ++j) {
            const int i = 64 * j + lane;
            *(i <= Nb ? s_indptr + i : s_spare) = ip[j];
        }
    }
#pragma unroll
    for (int u = 0; u < kBiasPer; ++u) {
        const int i = threadIdx.x + u * kThreads;
        *(i < Nb * R ? reinterpret_cast<int *>(s_bias) + i : s_spare) = __float_as_int(bv[u]);
    }
    for (int i = threadIdx.x + kBiasPer * kThreads; i < Nb * R; i += kThreads)
        s_bias[i] = bias ? bias[i] : 0.0f;

    if (lane_words >= 64 * kStageChunks)
        x_store(0, NoClamp{});
    else
        x_store(0, Clamp{});
    for (int c0 = 64 * kStageChunks; c0 < lane_words; c0 += 64 * kStageChunks) {
        x_load(c0);
        x_store(c0, Clamp{});
    }
    if constexpr (U::kPad == 1) {   // the fp32 R x 1 tile's zero pad column
        if (threadIdx.x < kTT) Xs[threadIdx.x * XP + K] = 0.0f;
    }
    if constexpr (U::kTransposed) {   // the transposed tile's zero pad column K
        if (threadIdx.x < kTT) reinterpret_cast<bf16_t *>(Xs)[K * XP + threadIdx.x] = 0;
    }
    __syncthreads();

    // Per-wave LDS scratch of units that stage their blocks (transposed bf16 32x1).
    char *wslot = reinterpret_cast<char *>(Xs) + I.wbuf_offset + wave * 2048;
    TileOut out;
    out.ldy4 = int(ldy) * 4;
    out.rsrc = buffer_rsrc(Y + t0 * ldy, unsigned(rows) * unsigned(out.ldy4));

    // Empty owned rows: Y = bias.  (The stream below visits only segments with blocks.)
    for (int r = rlo; r < rhi; ++r) {
        if (uniform(s_indptr[r + 1]) == uniform(s_indptr[r])) {
            typename U::Acc z;
            U::init(z, s_bias, r * R);
            U::store(z, out, r * R);
        }
    }

    // The wave's block range [Pw, Pw1) is cut into row segments: the head segment
    // [Pw, head_end) of row rlo - 1 (if any), then each owned row with blocks, clipped to Pw1.
    // Each segment is a counted loop over units of KB blocks from its start (the last one may
    // be partial, masked branch-free).  Operands are double-buffered in A/B: every unit's
    // MFMAs are issued after the loads of the following unit, which for a segment's last unit
    // is the first unit of the next segment.  Row bookkeeping (stores, zeroing) stays outside
    // the inner loop so the accumulator is updated in place.  An owned row's accumulator starts
    // at the bias; a head (a row another wave finishes) starts at zero.
    constexpr int KB = U::KB;
    typename U::Acc acc, head;
    U::zero(head);
    int tail_row = -1;

    if (has_head) {
        U::zero(acc);
    } else {
        if (row < rhi) U::init(acc, s_bias, row * R);
        else U::zero(acc);
    }
    if (row < rhi) {
        while (true) {
            int np, nend;
            const int nrow = next_row(row, np, nend);
            const bool more = nrow < rhi;
            // After the segment's last unit, prefetch the next segment's first unit (or, at
            // the very end, reload the current unit: a harmless in-bounds load).
            const int fp = more ? np : p;
            const int nu = (end - p + KB - 1) / KB;
            bool next_in_b;
            int u = 0;
            // sched_barrier keeps the compiler from sinking each prefetch next to its use,
            // which would leave no load in flight while the MFMAs run.  A partial last unit
            // has its operand registers masked (never the accumulator, which stays in place).
            while (true) {
                const int q = p + u * KB;
                const bool last = u + 1 == nu;
                U::load(B, last ? fp : q + KB, nnzb, indices, data);
                __builtin_amdgcn_sched_barrier(0);
                if (q + KB > end) U::mask(A, end - q);
                U::mma(acc, A, Xs, XP, Kb, wslot);
                __builtin_amdgcn_sched_barrier(0);
                if (last) {
                    next_in_b = true;
                    break;
                }
                ++u;
                const int q2 = p + u * KB;
                const bool last2 = u + 1 == nu;
                U::load(A, last2 ? fp : q2 + KB, nnzb, indices, data);
                __builtin_amdgcn_sched_barrier(0);
                if (q2 + KB > end) U::mask(B, end - q2);
                U::mma(acc, B, Xs, XP, Kb, wslot);
                __builtin_amdgcn_sched_barrier(0);
                if (last2) {
                    next_in_b = false;
                    break;
                }
                ++u;
            }
            // Finish the segment: head -> `head`, complete row -> Y, a row continuing past
            // Pw1 (necessarily the last segment) -> tail, left in `acc`.  The next segment is
            // an owned row.
            if (row == rlo - 1) {
                head = acc;
            } else if (uniform(s_indptr[row + 1]) <= Pw1) {
                U::store(acc, out, row * R);
            } else {
                tail_row = row;
            }
            if (!more) break;
            U::init(acc, s_bias, nrow * R);
            if (next_in_b) A = B;
            row = nrow;
            p = np;
            end = nend;
        }
    }

    // Combine rows cut by wave boundaries, in wave order: the owner's partial (bias and its
    // blocks), then each later wave's head partial.  The X tile is dead now; its LDS holds the
    // head partials P[w][v][lane], the partials of wide tails T[w][v][lane] and one word per
    // wave naming its wide tail row.  A tail with at most kLocalHeads heads is finished by its
    // owner; a wider one (a long row spread over many waves) is reduced by all waves at once,
    // wave v summing accumulator register v of every lane.
    constexpr int kLocalHeads = 2;
    constexpr int kSlot = U::kRegs * 64;   // floats per partial
    __syncthreads();
    float *P = reinterpret_cast<float *>(Xs);
    float *Tw = P + NW * kSlot;
    int *s_wide = reinterpret_cast<int *>(Tw + NW * kSlot);   // [NW] rows, then [NW] head masks
    // The waves holding head partials of the tail row this wave owns (bit w2 set): later waves
    // whose range starts before the row's end, except waves with an empty range.
    unsigned tail_heads = 0;
    if (tail_row >= 0) {
        const int e = uniform(s_indptr[tail_row + 1]);
        tail_heads = unsigned(__ballot(lane > wave && lane < NW && ws < e && wsn != ws));
    }
    const bool wide = __popc(tail_heads) > kLocalHeads;
    if (has_head) {
#pragma unroll
        for (int v = 0; v < U::kRegs; ++v) P[(wave * U::kRegs + v) * 64 + lane] = U::get(head, v);
    }
    if (wide) {
#pragma unroll
        for (int v = 0; v < U::kRegs; ++v) Tw[(wave * U::kRegs + v) * 64 + lane] = U::get(acc, v);
    }
    s_wide[wave] = wide ? tail_row : -1;
    s_wide[NW + wave] = int(tail_heads);
    __syncthreads();
    if (tail_row >= 0 && !wide) {
        for (unsigned m = tail_heads; m; m &= m - 1) {
            const int w2 = __ffs(m) - 1;
            float h[U::kRegs];
#pragma unroll
            for (int v = 0; v < U::kRegs; ++v) h[v] = P[(w2 * U::kRegs + v) * 64 + lane];
#pragma unroll
            for (int v = 0; v < U::kRegs; ++v) U::add(acc, v, h[v]);
        }
        U::store(acc, out, tail_row * R);
    }
    // Wide tails, in owner order.  All reads of a tail are issued before the sums; an absent
    // head adds -0, which leaves every value (also +0) unchanged.
    const int wv = lane < NW ? s_wide[lane] : -1;
    const int whm = lane < NW ? s_wide[NW + lane] : 0;
    for (unsigned long long m = __ballot(wv >= 0); m; m &= m - 1) {
        const int w = __ffsll(static_cast<long long>(m)) - 1;
        const int trow = __builtin_amdgcn_readlane(wv, w);
        if (wave < U::kRegs) {
            const unsigned hm = unsigned(__builtin_amdgcn_readlane(whm, w));
            const int v = wave;
            float x = Tw[(w * U::kRegs + v) * 64 + lane];
            float h[NW - 1];
#pragma unroll
            for (int i = 0; i < NW - 1; ++i) {
                const int w2 = i + 1;
                h[i] = P[(w2 * U::kRegs + v) * 64 + lane];
            }
#pragma unroll
            for (int i = 0; i < NW - 1; ++i) x += (hm >> (i + 1)) & 1u ? h[i] : -0.0f;
            U::store_reg(x, out, trow * R, v);
        }
    }
}

template <int R, int C, int NW, bool BF, int W = 1>
bsr_status launch_variant(const TiledBatch &batch, dim3 grid, size_t lds, hipStream_t st,
                          const LaunchEvents &ev) {
    launch_kernel(spmm_tiled_kernel<R, C, NW, BF, W>, grid, dim3(NW * 64), lds, st, ev, batch);
    return launch_status();
}

}  // namespace

bool wide_units(const TiledWork *work, int n) {
    int64_t blocks = 0, rows = 0;
    for (int i = 0; i < n; ++i) {
        blocks += work[i].W->nnzb;
        rows += work[i].W->n_rows / work[i].W->R;
    }
    return blocks >= kWideUnitRowBlocks * rows;
}

bool tiled_supported(int R, int C, int dtype) {
    if (dtype != BSR_F32 && dtype != BSR_BF16) return false;
    return (R == 32 && C == 1) || (R == 16 && C == 1) || (R == 32 && C == 32) ||
           (R == 16 && C == 16);
}

// Waves per workgroup, chosen so that each variant's registers fit without spilling
// (512 VGPRs per SIMD lane shared by the waves on that SIMD).
int tiled_waves(int R, int C) { return 16; }

TiledPlan plan_tiled(const void *X, int64_t T, int64_t ldx, const bsr_matrix_t *W, int64_t ldy,
                     int slices, size_t lds_limit) {
    TiledPlan p{};
    const int R = W->R, C = W->C;
    if (!tiled_supported(R, C, W->dtype)) return p;
    const int64_t K = W->n_cols, Nb = W->n_rows / R;
    const bool bf = W->dtype == BSR_BF16;
    const bool transposed = bf && R == 32 && C == 1;   // Unit<32, 1, true>::kTransposed
    const bool tile_bf16 = bf && (C > 1 || transposed);   // Unit<R, C, BF>::kTileBF16
    const int regs = (R == 32) ? 16 : 8;
    const int NW = tiled_waves(R, C);
    // Row pointers: indptr (square blocks); the unit row pointer and indptr (R x 1 blocks).
    p.ib_offset = C == 1 ? int((Nb + 1 + 3) & ~int64_t(3)) : 0;
    p.indptr_words = int((Nb + 1 + 3) & ~int64_t(3)) + p.ib_offset + 4;   // + a spare word
    p.bias_words = int((W->n_rows + 3) & ~int64_t(3));
    size_t tile_bytes;
    // Partials and wide tails of the combine (an accumulator of two token halves is combined
    // one half at a time, so `regs` per pass either way).
    const size_t h_bytes = 2 * size_t(NW) * regs * 64 * 4 + size_t(NW) * 8;
    const size_t head_bytes = size_t(p.indptr_words + p.bias_words) * 4;
    if (transposed) {
        // K + 1 columns (the last is the zero pad) of 32 tokens, pitch 36 bf16 (72 bytes,
        // 8-byte aligned for the transpose reads), then 2 KB of block scratch per wave.  With
        // many tokens the tile holds 64 tokens as two such halves one after the other: a unit's
        // weights then feed two matrix-core instructions (flat kernel only, TiledPlan::tokens).
        // 64-token tiles are taken when block-rows hold at least kTile64RowBlocks stored blocks
        // on average, there are at least 32 tiles (with slices they still give every CU an
        // item), Y's 64-row window stays below 2^31 bytes and LDS holds them.
        p.x_pitch = 36;
        const int64_t tiles64 = (T + 63) / 64;
        const size_t wbuf64 = size_t(((2 * (K + 1)) * 72 + 255) & ~int64_t(255));
        const size_t t64 = wbuf64 + size_t(NW) * 2048;
        if (R == 32 && C == 1 && W->nnzb >= kTile64RowBlocks * Nb && tiles64 >= 32 &&
            ldy < (int64_t(1) << 23) &&
            head_bytes + (t64 > h_bytes ? t64 : h_bytes) <= lds_limit) {
            p.tokens = 64;
            p.wbuf_offset = int(wbuf64);
            tile_bytes = t64;
        } else {
            p.wbuf_offset = int(((K + 1) * 72 + 255) & ~int64_t(255));
            tile_bytes = size_t(p.wbuf_offset) + size_t(NW) * 2048;
        }
    } else {
        p.x_pitch = int(tile_pitch(R, C, tile_bf16, K));
        p.wbuf_offset = 0;
        tile_bytes = size_t(kTT) * size_t(p.x_pitch) * (tile_bf16 ? 2 : 4);
    }
    p.lds_bytes = head_bytes + (tile_bytes > h_bytes ? tile_bytes : h_bytes);
    if (p.lds_bytes > lds_limit) return TiledPlan{};
    // Buffer ranges are 32-bit: the block data, one X row and a 32-row tile of Y stay below
    // 2^31 bytes.
    if (W->nnzb * R * C >= (int64_t(1) << 29)) return TiledPlan{};
    if (ldy >= (int64_t(1) << 24) || K >= (int64_t(1) << 24)) return TiledPlan{};
    // Square kernels read 8- or 16-byte vectors from data.
    const bool data_al = (reinterpret_cast<uintptr_t>(W->data) & 15) == 0;
    if (C > 1 && !data_al) return TiledPlan{};
    // bf16 X rows are read from their byte offset ldx * 2; keep them 4-byte aligned for the
    // dword loads of the bf16 tile.
    if (bf && C > 1 && ((reinterpret_cast<uintptr_t>(X) & 3) != 0 || (ldx & 1) != 0))
        return TiledPlan{};
    p.num_tiles = int((T + p.tokens - 1) / p.tokens);
    p.slices = slices > 0 ? slices : 1;
    if (p.slices > Nb) p.slices = int(Nb);
    p.ok = true;
    return p;
}

bsr_status launch_spmm_tiled(const TiledWork *work, int n, void *stream,
                             const LaunchEvents &ev) {
    if (n < 1 || n > kMaxItems) return BSR_ERR_ARG;
    const int R = work[0].W->R, C = work[0].W->C;
    TiledBatch batch{};
    batch.n = n;
    int gx = 0;   // workgroups per product: the largest product's pairs, rounded up to 8
    size_t lds = 0;
    for (int i = 0; i < n; ++i) {
        const TiledWork &w = work[i];
        if (w.W->R != R || w.W->C != C || w.W->dtype != work[0].W->dtype) return BSR_ERR_ARG;
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
        it.indptr_words = w.plan.indptr_words;
        it.bias_words = w.plan.bias_words;
        it.wbuf_offset = w.plan.wbuf_offset;
        it.ib_offset = w.plan.ib_offset;
        const int wgs = ((w.plan.num_tiles * w.plan.slices + 7) / 8) * 8;
        if (wgs > gx) gx = wgs;
        if (w.plan.lds_bytes > lds) lds = w.plan.lds_bytes;
    }
    hipStream_t st = as_stream(stream);
    if (R == 16 && C == 16 && wide_units(work, n)) {
        if (work[0].W->dtype == BSR_BF16)
            return launch_variant<16, 16, 16, true, 4>(batch, dim3(gx, n), lds, st, ev);
        return launch_variant<16, 16, 16, false, 4>(batch, dim3(gx, n), lds, st, ev);
    }
    // Linear R x 1 blocks run on the flat-stream kernel (spmm_flat.hip).
    if (work[0].W->dtype == BSR_BF16) {
        if (R == 32 && C == 32) return launch_variant<32, 32, 16, true>(batch, dim3(gx, n), lds, st, ev);
        if (R == 16 && C == 16) return launch_variant<16, 16, 16, true>(batch, dim3(gx, n), lds, st, ev);
    } else {
        if (R == 32 && C == 32) return launch_variant<32, 32, 16, false>(batch, dim3(gx, n), lds, st, ev);
        if (R == 16 && C == 16) return launch_variant<16, 16, 16, false>(batch, dim3(gx, n), lds, st, ev);
    }
    return BSR_ERR_UNSUPPORTED;
}

}  // namespace bsr
