// BSR product for linear R x 1 blocks (32x1, 16x1; fp32 or bf16 inputs, fp32 accumulate) on
// gfx950 matrix cores, as one flat stream of units per wave.
//
// Y[t][n] = bias[n] + sum over stored blocks p of block-row i = n / R of
//           X[t][indices[p]] * data[p][n - iR]                                       (Sec. 2.2)
//
// Once the input columns named by a block-row's indices are gathered, the row times a token
// tile is a small dense product whose contraction index is the block; the units of
// spmm_units.h run it on MFMA.  This kernel differs from the square-block tiled kernel in how
// a wave walks its work:
//   * every block-row is cut into units of KB consecutive stored blocks from its first block
//     (the last unit of a row is partial: its missing blocks read the tile's zero column with
//     zero weights), and rows are numbered in units by a row pointer over units, uptr;
//   * slices (whole block-rows) and the waves' shares inside a slice are balanced by units, so
//     a wave's share starts and ends on unit boundaries and no unit is cut by a wave boundary;
//   * a wave walks its units as one flat stream, row ends included, with the operands of the
//     next kDepth units in flight while it multiplies the current one (a ring of kDepth + 1
//     register buffers);
//   * the operands come either from the BSR arrays (indices, data; uptr computed in the
//     prologue from indptr) or from a plan prepared once per matrix (uptr, and every unit's
//     columns and weights packed in lane order: two 16-byte loads per lane and unit).  Both
//     give the same instructions on the same values, so Y is bit-identical with or without a
//     plan.
// The X tile staging, the bias, the combine of block-rows cut by wave boundaries (in wave
// order, in LDS) and the stores are those of the tiled kernel.
#include <climits>
#include <type_traits>

#include "device_common.h"
#include "spmm_tiled.h"
#include "spmm_units.h"

namespace bsr {

namespace {

constexpr int kNW = 16;            // waves per workgroup
// Units in flight ahead of the one being multiplied, per operand source (a split unit holds
// 16 blocks and six MFMAs, and its operands take 16 registers per lane), and the operand
// buffers per wave.
template <int PK>
constexpr int kDepthOf = PK == 2 ? 2 : 3;
template <int PK>
constexpr int kRingOf = kDepthOf<PK> + 1;
// 64-column X chunks a persistent workgroup prefetches per row (fewer for split units, whose
// operands need more registers).
template <int PK>
constexpr int kXChunksPersistent = PK == 2 ? 8 : 16;

// A slice's units are shared out over the 16 waves by weights that depend on a wave's place
// among the four waves of its SIMD (wave w runs on SIMD w % 4, after waves w - 4, w - 8, ...).
// The SIMDs' instruction arbitration favours older waves: with equal shares the first wave of
// every SIMD finished its stream about 30% before the last (per-wave timestamps on MI355X, the
// BERT-large 32x1 stack), and the item waits for the last.  Weights 48:38:31:27 made that
// launch 2% faster than equal shares (same box, A/B).  Start of wave l's units (l = 16: the end
// of the range).
constexpr unsigned kShareWeight[4] = {48, 38, 31, 27};
constexpr unsigned kShareTotal = 4 * (kShareWeight[0] + kShareWeight[1] + kShareWeight[2] +
                                      kShareWeight[3]);
__device__ __forceinline__ int wave_start(int64_t Q0, unsigned span, unsigned l) {
    const unsigned a = l >> 2, b = l & 3;
    unsigned cum = 0;
#pragma unroll
    for (unsigned i = 0; i < 4; ++i) cum += i < a ? 4 * kShareWeight[i] : 0u;
#pragma unroll
    for (unsigned i = 0; i < 4; ++i) cum += i == a ? b * kShareWeight[i] : 0u;
    return int(Q0) + int(uint64_t(span) * cum / kShareTotal);
}

// Inclusive prefix sum over the 64 lanes of a wave: row shifts by 1, 2, 4 and 8 lanes sum each
// row of 16 lanes, then the last lane of row 0 is added to row 1 and of row 2 to row 3, and
// the last lane of row 1 (now rows 0 and 1) to rows 2 and 3.  Lanes a shift reads from
// outside their row contribute 0.
__device__ __forceinline__ int wave_scan_incl(int v) {
    v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, false);   // row_shr:1
    v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, false);   // row_shr:2
    v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, false);   // row_shr:4
    v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, false);   // row_shr:8
    v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xa, 0xf, false);   // row_bcast:15
    v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xc, 0xf, false);   // row_bcast:31
    return v;
}

// Empty owned rows, the stream and the combine of one (token tile, slice) item, shared by the
// one-item and the persistent kernel.  `it` holds the wave's share and the LDS layout; the
// ring holds the operands of the share's first kDepth units; fetch(ops, nvalid, u) loads
// unit u (nothing past the share).
struct FlatItem {
    int lane, wave;
    int Pw, Pw1;        // the wave's units
    int rlo, rhi;       // the rows it owns
    int row, end;       // first row piece: its row and the end of its units
    bool has_head;      // the share starts inside row rlo - 1
    int ws, wsn;        // wave starts, one per lane: wave `lane` and wave lane + 1
    const int *s_up;    // unit row pointer (LDS)
    const float *s_bias;
    float *Xs;          // X tile (LDS), reused by the combine
    int XP, Kb;
    char *wslot;
    TileOut out;
    // Paired products: rows from rsplit on belong to the second product, whose Y tile is out2
    // (its rows counted from rsplit); rsplit = INT_MAX without a pair.
    TileOut out2;
    int rsplit;
};

// The tile and accumulator of a launch (TT tokens per tile: 64 only for bf16 32x1 blocks) and
// the operand source of a unit: the BSR arrays (PK = 0), a native plan (1) or a split plan (2).
template <int R, bool BF, int TT>
using TileOf = std::conditional_t<TT == 64, Unit64BF, Unit<R, 1, BF>>;
template <int R, bool BF, int PK, int TT>
using SrcOf = std::conditional_t<
    PK == 2, SplitPlanUnit,
    std::conditional_t<PK == 1, std::conditional_t<TT == 64, PlanUnit64BF, PlanUnit<R, 1, BF>>,
                       TileOf<R, BF, TT>>>;

template <int R, bool BF, int PK, int TT, bool PAIR = false, class Ops, class Fetch>
__device__ __forceinline__ void flat_item_body(const FlatItem &it, Ops (&ring)[kRingOf<PK>],
                                               int (&nvr)[kRingOf<PK>], Fetch &&fetch) {
    using U = TileOf<R, BF, TT>;
    using Src = SrcOf<R, BF, PK, TT>;
    constexpr bool PL = PK != 0;
    constexpr int kDepth = kDepthOf<PK>, kRing = kRingOf<PK>;
    constexpr int NW = kNW, KB = U::KB;
    const int lane = it.lane, wave = it.wave, Pw = it.Pw, Pw1 = it.Pw1, rlo = it.rlo,
              rhi = it.rhi, XP = it.XP, Kb = it.Kb, ws = it.ws, wsn = it.wsn;
    const bool has_head = it.has_head;
    const int *s_up = it.s_up;
    const float *s_bias = it.s_bias;
    float *Xs = it.Xs;
    char *wslot = it.wslot;
    const TileOut &out = it.out;
    int r = it.row;
    int r_end = it.end;
    // The Y tile of row rr and the row's first output column in it.
    auto out_of = [&](int rr, int &n0) -> const TileOut & {
        if constexpr (PAIR) {
            if (rr >= it.rsplit) {
                n0 = (rr - it.rsplit) * R;
                return it.out2;
            }
        }
        n0 = rr * R;
        return out;
    };
    // Empty owned rows: Y = bias.
    for (int rr = rlo; rr < rhi; ++rr) {
        if (uniform(s_up[rr + 1]) == uniform(s_up[rr])) {
            typename U::Acc z;
            U::init(z, s_bias, rr * R);
            int n0;
            const TileOut &o = out_of(rr, n0);
            U::store(z, o, n0);
        }
    }

    // First row after r with units (rhi if none); returns its start and clipped end.
    auto next_row = [&](int rr, int &start, int &end_) -> int {
        for (++rr; rr < rhi; ++rr) {
            start = uniform(s_up[rr]);
            const int e = uniform(s_up[rr + 1]);
            if (start < e) {
                end_ = e < Pw1 ? e : Pw1;
                return rr;
            }
        }
        start = end_ = 0;
        return rhi;
    };

    // The stream.  Unit u is multiplied in ring slot (u - Pw) mod kRing, after the loads of
    // unit u + kDepth are issued into the slot freed by unit u - 1.  At the last unit of a row
    // piece the accumulator goes to Y (a complete row), to `head` (a row another wave finishes)
    // or stays as the tail (a row continuing past Pw1), and the next row starts at its bias.
    typename U::Acc acc, head;
    U::zero(head);
    int tail_row = -1;
    if (has_head) U::zero(acc);
    else if (r < rhi) U::init(acc, s_bias, r * R);
    else U::zero(acc);
    // Every phase issues its loads (past the wave's range they fetch nothing) and the loop
    // exits only at its top, so every path through the loop issues the same loads in the same
    // order: the compiler then counts kDepth units' loads between a unit's loads and its use
    // and waits for that unit alone.
    for (int base = Pw; base < Pw1; base += kRing) {
#pragma unroll
        for (int ph = 0; ph < kRing; ++ph) {
            const int u = base + ph;
            fetch(ring[(ph + kDepth) % kRing], nvr[(ph + kDepth) % kRing], u + kDepth);
            __builtin_amdgcn_sched_barrier(0);
            if (u >= Pw1) continue;
            if constexpr (!PL) {
                if (nvr[ph] < KB) U::mask(ring[ph], nvr[ph]);
            }
            typename Src::A xa;
            Src::gather(xa, ring[ph], Xs, XP, Kb, wslot);
            Src::mac(acc, xa, ring[ph]);
            __builtin_amdgcn_sched_barrier(0);
            if (u + 1 == r_end) {
                if (r == rlo - 1) {
                    head = acc;
                } else if (uniform(s_up[r + 1]) <= Pw1) {
                    int n0;
                    const TileOut &o = out_of(r, n0);
                    U::store(acc, o, n0);
                } else {
                    tail_row = r;
                }
                int np, nend;
                r = next_row(r, np, nend);
                r_end = nend;
                if (r < rhi) U::init(acc, s_bias, r * R);
            }
        }
    }

    // Combine rows cut by wave boundaries, in wave order (as in the tiled kernel): the owner's
    // partial (bias and its units), then each later wave's head partial.  The X tile is dead
    // now; its LDS holds the head partials P[w][v][lane], the partials of wide tails
    // T[w][v][lane] and one word per wave naming its wide tail row.  An accumulator of two
    // 32-token halves is combined in two passes, one half (16 registers) per pass.
    constexpr int kLocalHeads = 2;
    constexpr int kPassRegs = U::kRegs / U::kHalves;
    constexpr int kSlot = kPassRegs * 64;
    float *P = reinterpret_cast<float *>(Xs);
    float *Tw = P + NW * kSlot;
    int *s_wide = reinterpret_cast<int *>(Tw + NW * kSlot);
    unsigned tail_heads = 0;
    if (tail_row >= 0) {
        const int e = uniform(s_up[tail_row + 1]);
        tail_heads = unsigned(__ballot(lane > wave && lane < NW && ws < e && wsn != ws));
    }
    const bool wide = __popc(tail_heads) > kLocalHeads;
#pragma unroll
    for (int hh = 0; hh < U::kHalves; ++hh) {
        const int v0 = hh * kPassRegs;
        __syncthreads();   // the X tile (first pass) or the previous pass's partials are dead
        if (has_head) {
#pragma unroll
            for (int vv = 0; vv < kPassRegs; ++vv)
                P[(wave * kPassRegs + vv) * 64 + lane] = U::get(head, v0 + vv);
        }
        if (wide) {
#pragma unroll
            for (int vv = 0; vv < kPassRegs; ++vv)
                Tw[(wave * kPassRegs + vv) * 64 + lane] = U::get(acc, v0 + vv);
        }
        if (hh == 0) {
            s_wide[wave] = wide ? tail_row : -1;
            s_wide[NW + wave] = int(tail_heads);
        }
        __syncthreads();
        if (tail_row >= 0 && !wide) {
            for (unsigned m = tail_heads; m; m &= m - 1) {
                const int w2 = __ffs(m) - 1;
                float h[kPassRegs];
#pragma unroll
                for (int vv = 0; vv < kPassRegs; ++vv) h[vv] = P[(w2 * kPassRegs + vv) * 64 + lane];
#pragma unroll
                for (int vv = 0; vv < kPassRegs; ++vv) U::add(acc, v0 + vv, h[vv]);
            }
            int n0;
            const TileOut &o = out_of(tail_row, n0);
            if constexpr (U::kHalves == 1) U::store(acc, o, n0);
            else U::store_half(acc, o, n0, hh);
        }
        const int wv = lane < NW ? s_wide[lane] : -1;
        const int whm = lane < NW ? s_wide[NW + lane] : 0;
        for (unsigned long long m = __ballot(wv >= 0); m; m &= m - 1) {
            const int w = __ffsll(static_cast<long long>(m)) - 1;
            const int trow = __builtin_amdgcn_readlane(wv, w);
            if (wave < kPassRegs) {
                const unsigned hm = unsigned(__builtin_amdgcn_readlane(whm, w));
                const int vv = wave;
                float x = Tw[(w * kPassRegs + vv) * 64 + lane];
                float h[NW - 1];
#pragma unroll
                for (int i = 0; i < NW - 1; ++i) h[i] = P[((i + 1) * kPassRegs + vv) * 64 + lane];
#pragma unroll
                for (int i = 0; i < NW - 1; ++i) x += (hm >> (i + 1)) & 1u ? h[i] : -0.0f;
                int n0;
                const TileOut &o = out_of(trow, n0);
                U::store_reg(x, o, n0, v0 + vv);
            }
        }
    }
}

template <int R, bool BF, int PK, int TT>
__global__ __launch_bounds__(kNW * 64) void spmm_flat_kernel(const TiledBatch batch) {
    using U = TileOf<R, BF, TT>;
    using Src = SrcOf<R, BF, PK, TT>;
    static_assert(U::kTokens == TT, "the unit's tile holds TT tokens");
    constexpr bool PL = PK != 0;
    constexpr int kDepth = kDepthOf<PK>, kRing = kRingOf<PK>;
    using Ops = typename Src::Ops;
    constexpr int NW = kNW, KB = U::KB, kThreads = NW * 64;
    extern __shared__ float smem[];

    const int lane = threadIdx.x & 63, wave = uniform(threadIdx.x >> 6);
    const int g = blockIdx.x;
    const TiledItem &I = batch.item[blockIdx.y];
    const void *__restrict__ X = I.X;
    const int64_t T = I.T, ldx = I.ldx, ldy = I.ldy;
    const int32_t *__restrict__ indptr = I.indptr;
    const int32_t *__restrict__ indices = I.indices;
    const void *__restrict__ data = I.data;
    const int32_t *__restrict__ uptr = I.uptr;
    const int32_t *__restrict__ ucol = I.ucol;
    const void *__restrict__ uval = I.uval;
    const float *__restrict__ bias = I.bias;
    float *__restrict__ Y = I.Y;
    const int K = I.K, nnzb = I.nnzb, Nb = I.Nb, Kb = I.Kb, num_tiles = I.num_tiles,
              slices = I.slices, XP = I.XP;
    // The largest unit position: a plan's reserved units, or (unplanned) nnzb, which bounds
    // the units computed from indptr (every unit holds at least one block).
    const int ucap = PL ? I.ucap : nnzb;
    // LDS: the unit row pointer s_up[Nb + 1], the block row pointer s_ib[Nb + 1] (unplanned),
    // a spare word, the bias, then the X tile (reused for partial tiles at the end).
    int *s_up = reinterpret_cast<int *>(smem);
    int *s_ib = s_up + I.ib_offset;
    float *s_bias = smem + I.indptr_words;
    float *Xs = s_bias + I.bias_words;

    asm volatile("" ::"s"(X), "s"(T), "s"(ldx), "s"(ldy), "s"(indptr), "s"(indices), "s"(data),
                 "s"(bias), "s"(Y));
    asm volatile("" ::"s"(K), "s"(nnzb), "s"(Nb), "s"(Kb), "s"(num_tiles), "s"(slices), "s"(XP),
                 "s"(I.indptr_words), "s"(I.bias_words), "s"(I.wbuf_offset));

    // Workgroup -> (token tile, slice), XCD-aware as in the tiled kernel: ids with equal
    // blockIdx.x mod 8 share an XCD; a product's (tile, slice) pairs in tile-major order are cut
    // into 8 contiguous ranges, one per XCD.
    const int xcd = g & 7, rank = g >> 3;
    const int pairs = num_tiles * slices, per_xcd = (pairs + 7) >> 3;
    const int q = xcd * per_xcd + rank;
    if (rank >= per_xcd || q >= pairs) return;
    const int tile = q / slices, s = q - tile * slices;
    const int64_t t0 = int64_t(tile) * TT;

    const int rows = int(T - t0 < TT ? T - t0 : TT);
    constexpr int kXBytes = BF ? 2 : 4;
    constexpr int kRowsPerWave = TT / NW;
    static_assert(TT % NW == 0, "every wave stages the same number of rows");
    // 64-column chunks of an X row staged per pass (the registers of a pass are the same for
    // both tile sizes).
    constexpr int kChunks = kStageChunks * 32 / TT;

    // Prologue, overlapping the latencies of the row pointers, the X tile and the first units:
    //   (1) every wave loads the row pointers into registers, the bias, then its X-tile rows;
    //   (2) it computes the unit row pointer (unplanned: from indptr, by a wave prefix sum),
    //       its share of the slice and issues its first units' loads;
    //   (3) row pointers, bias and the X tile go to LDS and one barrier ends the prologue.
    // A product with 256 or more block-rows copies the row pointers to LDS first.
    constexpr int kIpChunks = 4;   // row-pointer entries per wave in registers: 64 per chunk
    constexpr int kBiasPer = 4;    // bias entries per thread staged through registers
    const bool reg_part = Nb < 64 * kIpChunks;
    int up[kIpChunks];   // uptr[64 j + lane]
    int ib[kIpChunks];   // indptr[64 j + lane] (unplanned)
    float bv[kBiasPer];
    {
        const __amdgpu_buffer_rsrc_t rb = buffer_rsrc(bias, bias ? unsigned(Nb * R) * 4u : 0u);
        const unsigned off = reg_part ? unsigned(lane) * 4u : 0x7ffff000u;
        if constexpr (PL) {
            const __amdgpu_buffer_rsrc_t rup = buffer_rsrc(uptr, unsigned(Nb + 1) * 4u);
#pragma unroll
            for (int j = 0; j < kIpChunks; ++j)
                up[j] = __builtin_amdgcn_raw_buffer_load_b32(rup, off + 256 * j, 0, 0);
        } else {
            // indptr[i] and indptr[i + 1] per lane; a row's unit count is ceil(blocks / KB).
            const __amdgpu_buffer_rsrc_t rip = buffer_rsrc(indptr, unsigned(Nb + 1) * 4u);
            int ibn[kIpChunks];
#pragma unroll
            for (int j = 0; j < kIpChunks; ++j) {
                ib[j] = __builtin_amdgcn_raw_buffer_load_b32(rip, off + 256 * j, 0, 0);
                ibn[j] = __builtin_amdgcn_raw_buffer_load_b32(rip, off + 256 * j + 4, 0, 0);
            }
#pragma unroll
            for (int j = 0; j < kIpChunks; ++j) {
                ib[j] = clampi(ib[j], 0, nnzb);
                const int n = clampi(ibn[j], 0, nnzb) - ib[j];
                up[j] = (64 * j + lane < Nb && n > 0) ? (n + KB - 1) / KB : 0;
            }
        }
#pragma unroll
        for (int u = 0; u < kBiasPer; ++u)
            bv[u] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                                  rb, (threadIdx.x + u * kThreads) * 4, 0, 0));
    }

    // X tile staging (as in the tiled kernel): loads into v, then conflict-free LDS stores.
    constexpr int kColsPerLane = 1;
    const int lane_words = K;
    unsigned v[kRowsPerWave][kChunks];
    auto x_load = [&](int c0) {
#pragma unroll
        for (int r = 0; r < kRowsPerWave; ++r) {
            const int t = wave + NW * r;
            const int tr = t < rows ? t : rows - 1;
            const __amdgpu_buffer_rsrc_t rx =
                buffer_rsrc(static_cast<const char *>(X) + (t0 + tr) * ldx * kXBytes,
                            t < rows ? unsigned(K) * kXBytes : 0u);
#pragma unroll
            for (int m = 0; m < kChunks; ++m) {
                if constexpr (BF)
                    v[r][m] = __builtin_amdgcn_raw_buffer_load_b16(rx, (c0 + lane) * 2 + 128 * m,
                                                                   0, 0);
                else
                    v[r][m] = __builtin_amdgcn_raw_buffer_load_b32(rx, (c0 + lane) * 4 + 256 * m,
                                                                   0, 0);
            }
        }
    };
    auto x_store = [&](int c0, auto clamp) {
#pragma unroll
        for (int r = 0; r < kRowsPerWave; ++r) {
            const int t = wave + NW * r;
            if constexpr (U::kTransposed) {
                // Tokens 32 h .. 32 h + 31 go to half h of the transposed tile.
                bf16_t *xt = reinterpret_cast<bf16_t *>(Xs) + (t >> 5) * ((K + 1) * XP) + (t & 31);
#pragma unroll
                for (int m = 0; m < kChunks; ++m) {
                    const int c = c0 + 64 * m + lane;
                    xt[(decltype(clamp)::value ? min(c, K) : c) * XP] = bf16_t(v[r][m]);
                }
            } else {
                unsigned *dst = reinterpret_cast<unsigned *>(Xs) + t * XP;
#pragma unroll
                for (int m = 0; m < kChunks; ++m) {
                    unsigned w = v[r][m];
                    if constexpr (BF) w <<= 16;   // bf16 -> fp32, exact
                    const int c = c0 + 64 * m + lane;
                    dst[decltype(clamp)::value ? min(c, lane_words) : c] = w;
                }
            }
        }
    };
    static_assert(kColsPerLane == 1, "R x 1 tiles move one column per lane");
    using Clamp = std::true_type;
    using NoClamp = std::false_type;
    x_load(0);

    // The wave's share, in units.  Slice s covers whole block-rows [row_lo, row_hi), row_lo the
    // first row whose unit start is >= floor(s U / slices); its units [Q0, Q1) are split evenly
    // over the waves (wave w: [Pw, Pw1)).  A wave owns the rows whose first unit lies in its
    // range (the last wave also owns trailing empty rows); units at the front of its range that
    // belong to row rlo - 1 are a head, summed into that row by the wave that owns it.
    int64_t k, Q0, Q1;
    int row_lo, row_hi, Pw, Pw1, rlo, rhi, head_end, row, p, end;
    int ws = 0, wsn = 0;   // wave starts, one per lane: wave `lane` and wave lane + 1
    auto share = [&](auto lower_bound) {
        static_assert(NW == 16, "wave starts are weighted for 16 waves");
        const unsigned span = unsigned(Q1 - Q0);
        ws = wave_start(Q0, span, unsigned(lane));
        wsn = wave_start(Q0, span, unsigned(lane) + 1);
        Pw = __builtin_amdgcn_readlane(ws, wave);
        Pw1 = __builtin_amdgcn_readlane(wsn, wave);
        rlo = (wave == 0) ? row_lo : lower_bound(int64_t(Pw));
        rlo = rlo < row_lo ? row_lo : (rlo > row_hi ? row_hi : rlo);
        rhi = (wave == NW - 1) ? row_hi : lower_bound(int64_t(Pw1));
        rhi = rhi < rlo ? rlo : (rhi > row_hi ? row_hi : rhi);
    };
    // Entry i (uniform, <= Nb) of a register-resident row pointer: one lane read per chunk and
    // a scalar select.
    auto lane_read = [&](const int(&a)[kIpChunks], int i, auto nch) -> int {
        constexpr int NCH = decltype(nch)::value;
        const int l = i & 63, c = i >> 6;
        int x = __builtin_amdgcn_readlane(a[0], l);
#pragma unroll
        for (int j = 1; j < NCH; ++j) {
            const int y = __builtin_amdgcn_readlane(a[j], l);
            x = c == j ? y : x;
        }
        return x;
    };
    auto reg_partition = [&](auto nch) {
        constexpr int NCH = decltype(nch)::value;
        if constexpr (PL) {
#pragma unroll
            for (int j = 0; j < NCH; ++j) up[j] = clampi(up[j], 0, ucap);
        } else {
            // Exclusive prefix of the per-row unit counts, chunk by chunk.
            int carry = 0;
#pragma unroll
            for (int j = 0; j < NCH; ++j) {
                const int incl = wave_scan_incl(up[j]) + carry;
                const int excl = incl - up[j];
                carry = __builtin_amdgcn_readlane(incl, 63);
                up[j] = excl;
            }
        }
        unsigned long long in_rows[NCH];
#pragma unroll
        for (int j = 0; j < NCH; ++j) in_rows[j] = __ballot(64 * j + lane < Nb);
        auto count_rows = [&](auto pred) -> int {
            int c = 0;
#pragma unroll
            for (int j = 0; j < NCH; ++j) c += __popcll(__ballot(pred(up[j])) & in_rows[j]);
            return c;
        };
        k = lane_read(up, Nb, nch);
        auto slice_start = [&](int s2) -> int {
            const uint64_t sk = uint64_t(s2) * uint64_t(k);
            return count_rows([&](int x) { return uint64_t(x + 1) * uint64_t(slices) <= sk; });
        };
        row_lo = (s == 0) ? 0 : slice_start(s);
        row_hi = (s == slices - 1) ? Nb : slice_start(s + 1);
        Q0 = lane_read(up, row_lo, nch);
        Q1 = lane_read(up, row_hi, nch);
        if (Q1 < Q0) Q1 = Q0;
        share([&](int64_t v) { return count_rows([&](int x) { return x < int(v); }); });
        head_end = (rlo < rhi) ? lane_read(up, rlo, nch) : Pw1;
        head_end = head_end < Pw ? Pw : (head_end > Pw1 ? Pw1 : head_end);
        if (head_end > Pw) {
            row = rlo - 1;
            p = Pw;
            end = head_end;
        } else {
            // First owned row with units: the last row i with uptr[i] <= uptr[rlo], if its
            // units extend past that start.
            row = rhi;
            p = end = 0;
            if (rlo < rhi) {
                const int v0 = lane_read(up, rlo, nch);
                const int c = count_rows([&](int x) { return x < v0 + 1; });
                const int e = lane_read(up, c, nch);
                if (c - 1 >= rlo && c - 1 < rhi && e > v0) {
                    row = c - 1;
                    p = v0;
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
        // Row pointers in LDS; unplanned, wave 0 forms the unit row pointer by prefix sums.
        if constexpr (PL) {
            for (int i = threadIdx.x; i <= Nb; i += kThreads) s_up[i] = clampi(uptr[i], 0, ucap);
        } else {
            for (int i = threadIdx.x; i <= Nb; i += kThreads) s_ib[i] = clampi(indptr[i], 0, nnzb);
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
        if constexpr (!PL) {
            if (wave == 0) {
                int carry = 0;
                for (int base = 0; base <= Nb; base += 64) {
                    const int i = base + lane;
                    const int n = i < Nb ? s_ib[i + 1] - s_ib[i] : 0;
                    const int cnt = n > 0 ? (n + KB - 1) / KB : 0;
                    const int incl = wave_scan_incl(cnt) + carry;
                    if (i <= Nb) s_up[i] = incl - cnt;
                    carry = __builtin_amdgcn_readlane(incl, 63);
                }
            }
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
            __builtin_amdgcn_s_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
        }
        k = uniform(s_up[Nb]);
        row_lo = (s == 0) ? 0 : uniform(wave_lower_bound(s_up, Nb, int64_t(s) * k / slices));
        row_hi = (s == slices - 1)
                     ? Nb
                     : uniform(wave_lower_bound(s_up, Nb, int64_t(s + 1) * k / slices));
        Q0 = uniform(s_up[row_lo]);
        Q1 = uniform(s_up[row_hi]);
        if (Q1 < Q0) Q1 = Q0;
        share([&](int64_t v) { return uniform(wave_lower_bound(s_up, Nb, v)); });
        head_end = (rlo < rhi) ? uniform(s_up[rlo]) : Pw1;
        head_end = head_end < Pw ? Pw : (head_end > Pw1 ? Pw1 : head_end);
        row = rlo - 1;
        p = Pw;
        end = head_end;
        if (head_end <= Pw) {
            for (row = rlo; row < rhi; ++row) {
                p = uniform(s_up[row]);
                const int e = uniform(s_up[row + 1]);
                if (p < e) {
                    end = e < Pw1 ? e : Pw1;
                    break;
                }
            }
            if (row >= rhi) p = end = 0;
        }
    }
    const bool has_head = head_end > Pw;

    // Prefetch cursor (unplanned): the row of the next unit to load, its units [pr_u0, pr_u1)
    // and blocks [pr_b0, pr_b1).
    int pr = row, pr_u0 = 0, pr_u1 = 0, pr_b0 = 0, pr_b1 = 0;
    auto read_up_lds = [&](int i) { return uniform(s_up[i]); };
    auto read_ib_lds = [&](int i) { return uniform(s_ib[i]); };
    // Loads the operands of unit uu (units past the wave's range fetch nothing).
    auto fetch = [&](Ops &o, int &nvalid, int uu, auto readU, auto readB) {
        if constexpr (PL) {
            Src::load(o, uu, Pw1, ucol, uval);
            nvalid = KB;
        } else {
            int p0 = nnzb, nv = KB;
            if (uu < Pw1) {
                while (uu >= pr_u1 && pr < Nb - 1) {
                    ++pr;
                    pr_u0 = pr_u1;
                    pr_u1 = readU(pr + 1);
                    pr_b0 = readB(pr);
                    pr_b1 = readB(pr + 1);
                }
                p0 = pr_b0 + KB * (uu - pr_u0);
                p0 = p0 < nnzb ? p0 : nnzb;
                nv = pr_b1 - p0 < KB ? pr_b1 - p0 : KB;
            }
            U::load(o, p0, nnzb, indices, data);
            nvalid = nv;
        }
    };
    Ops ring[kRing];
    int nvr[kRing];
    // Prime the ring with the first kDepth units (issued under the X-tile stores).
    auto prime = [&](auto readU, auto readB) {
        if constexpr (!PL) {
            if (row < rhi) {
                pr_u0 = readU(row);
                pr_u1 = readU(row + 1);
                pr_b0 = readB(row);
                pr_b1 = readB(row + 1);
            }
        }
#pragma unroll
        for (int d = 0; d < kDepth; ++d) fetch(ring[d], nvr[d], Pw + d, readU, readB);
    };
    if (reg_part) {
        if (Nb < 64)
            prime([&](int i) { return lane_read(up, i, std::integral_constant<int, 1>{}); },
                  [&](int i) { return lane_read(ib, i, std::integral_constant<int, 1>{}); });
        else
            prime([&](int i) { return lane_read(up, i, std::integral_constant<int, kIpChunks>{}); },
                  [&](int i) { return lane_read(ib, i, std::integral_constant<int, kIpChunks>{}); });
    } else {
        prime(read_up_lds, read_ib_lds);
    }

    // Row pointers (register path: wave 0) and bias into LDS.  Threads past the arrays write a
    // spare word at the end of the row-pointer region.
    int *s_spare = s_up + I.indptr_words - 1;
    if (reg_part && wave == 0) {
#pragma unroll
        for (int j = 0; j < kIpChunks; ++j) {
            const int i = 64 * j + lane;
            *(i <= Nb ? s_up + i : s_spare) = up[j];
            if constexpr (!PL) *(i <= Nb ? s_ib + i : s_spare) = ib[j];
        }
    }
#pragma unroll
    for (int u = 0; u < kBiasPer; ++u) {
        const int i = threadIdx.x + u * kThreads;
        *(i < Nb * R ? reinterpret_cast<int *>(s_bias) + i : s_spare) = __float_as_int(bv[u]);
    }
    for (int i = threadIdx.x + kBiasPer * kThreads; i < Nb * R; i += kThreads)
        s_bias[i] = bias ? bias[i] : 0.0f;

    if (lane_words >= 64 * kChunks)
        x_store(0, NoClamp{});
    else
        x_store(0, Clamp{});
    for (int c0 = 64 * kChunks; c0 < lane_words; c0 += 64 * kChunks) {
        x_load(c0);
        x_store(c0, Clamp{});
    }
    if constexpr (U::kPad == 1) {   // the fp32 tile's zero pad column
        if (threadIdx.x < TT) Xs[threadIdx.x * XP + K] = 0.0f;
    }
    if constexpr (U::kTransposed) {   // the transposed tile's zero pad column K
        if (threadIdx.x < TT)
            reinterpret_cast<bf16_t *>(Xs)[(threadIdx.x >> 5) * ((K + 1) * XP) + K * XP +
                                           (threadIdx.x & 31)] = 0;
    }
    __syncthreads();

    FlatItem fi{lane, wave, Pw, Pw1, rlo, rhi, row, end, has_head, ws, wsn, s_up, s_bias, Xs,
                XP, Kb, reinterpret_cast<char *>(Xs) + I.wbuf_offset + wave * 2048, TileOut{},
                TileOut{}, INT_MAX};
    fi.out.ldy4 = int(ldy) * 4;
    fi.out.rsrc = buffer_rsrc(Y + t0 * ldy, unsigned(rows) * unsigned(fi.out.ldy4));
    flat_item_body<R, BF, PK, TT>(fi, ring, nvr, [&](Ops &o, int &nv, int uu) {
        fetch(o, nv, uu, read_up_lds, read_ib_lds);
    });
}

// The persistent form: one workgroup per CU, each walking several (token tile, slice) items of
// its product, used when a launch has more items than the GPU has CUs.  The row pointers and
// the bias go to LDS once; every item then stores its X tile from registers (loaded under the
// previous item's stream), computes its wave's share from the LDS row pointers, issues its
// first units' loads, and after one barrier loads the next item's X rows into registers and
// runs the shared stream and combine.  Items of one workgroup share an XCD, as in the one-item
// kernel's mapping.
//
// PAIR (planned products only): the workgroups of group blockIdx.y serve two products that share
// X (the same token tiles), item.partner naming the second.  An item then covers both
// products' block-rows for one X tile: the rows of the second follow those of the first (its
// units after the first's), so one X store, one share computation and one combine serve twice
// the work, and the waves' shares run across the boundary.
template <int R, bool BF, int PK, int TT, bool PAIR = false>
__global__ __launch_bounds__(kNW * 64) void spmm_flat_persistent_kernel(const TiledBatch batch) {
    using U = TileOf<R, BF, TT>;
    using Src = SrcOf<R, BF, PK, TT>;
    static_assert(U::kTokens == TT, "the unit's tile holds TT tokens");
    constexpr bool PL = PK != 0;
    constexpr int kDepth = kDepthOf<PK>, kRing = kRingOf<PK>;
    using Ops = typename Src::Ops;
    constexpr int NW = kNW, KB = U::KB, kThreads = NW * 64;
    extern __shared__ float smem[];

    const int lane = threadIdx.x & 63, wave = uniform(threadIdx.x >> 6);
    const int g = blockIdx.x;
    const TiledItem &I = batch.item[blockIdx.y];
    static_assert(!PAIR || PK != 0, "paired products are planned");
    const TiledItem &IB = batch.item[PAIR ? I.partner : blockIdx.y];   // the second product
    const void *__restrict__ X = I.X;
    const int64_t T = I.T, ldx = I.ldx, ldy = I.ldy;
    const int32_t *__restrict__ indptr = I.indptr;
    const int32_t *__restrict__ indices = I.indices;
    const void *__restrict__ data = I.data;
    const int32_t *__restrict__ uptr = I.uptr;
    const int32_t *__restrict__ ucol = I.ucol;
    const void *__restrict__ uval = I.uval;
    const float *__restrict__ bias = I.bias;
    float *__restrict__ Y = I.Y;
    // Nb: the item's block-rows (both products' when paired; the second's follow NbA).
    const int NbA = I.Nb;
    const int K = I.K, nnzb = I.nnzb, Nb = PAIR ? I.Nb + IB.Nb : I.Nb, Kb = I.Kb,
              num_tiles = I.num_tiles, slices = I.slices, XP = I.XP;
    const int ucap = PL ? I.ucap : nnzb;
    int *s_up = reinterpret_cast<int *>(smem);
    int *s_ib = s_up + I.ib_offset;
    float *s_bias = smem + I.indptr_words;
    float *Xs = s_bias + I.bias_words;

    // Items: the XCD's range of the product's (tile, slice) pairs, round robin over the
    // gridDim.x / 8 workgroups of the XCD.
    const int xcd = g & 7, rank = g >> 3, nrank = int(gridDim.x) >> 3;
    const int pairs = num_tiles * slices, per_xcd = (pairs + 7) >> 3;
    const int q_first = xcd * per_xcd + rank;
    const int q_end = min(xcd * per_xcd + per_xcd, pairs);
    if (q_first >= q_end) return;

    constexpr int kXBytes = BF ? 2 : 4;
    constexpr int kRowsPerWave = TT / NW;
    constexpr int kXC = kXChunksPersistent<PK> * 32 / TT;
    static_assert(TT % NW == 0, "every wave stages the same number of rows");

    // X rows w + 16 r of a tile in registers, kXC 64-column chunks from column c0.  Rows past
    // the product's last token, and a tile of no rows (the prefetch after the last item), load
    // zeros from an empty buffer range.  A guarded load skips chunks that start at or past K;
    // the prefetch is unguarded, so that every path issues the same loads and the waits in the
    // stream count them.
    unsigned v[kRowsPerWave][kXC];
    auto x_load = [&](int64_t t0_, int rows_, int c0, bool guarded) {
#pragma unroll
        for (int r = 0; r < kRowsPerWave; ++r) {
            const int t = wave + NW * r;
            const int64_t row = t < rows_ ? t0_ + t : 0;
            const __amdgpu_buffer_rsrc_t rx =
                buffer_rsrc(static_cast<const char *>(X) + row * ldx * kXBytes,
                            t < rows_ ? unsigned(K) * kXBytes : 0u);
#pragma unroll
            for (int m = 0; m < kXC; ++m) {
                if (guarded && c0 + 64 * m >= K) continue;
                if constexpr (BF)
                    v[r][m] = __builtin_amdgcn_raw_buffer_load_b16(rx, (c0 + lane) * 2 + 128 * m,
                                                                   0, 0);
                else
                    v[r][m] = __builtin_amdgcn_raw_buffer_load_b32(rx, (c0 + lane) * 4 + 256 * m,
                                                                   0, 0);
            }
        }
    };
    // Chunks that start at or past K are not stored; a chunk that crosses K sends its columns
    // past K to column K, the tile's zero pad column.  The lane index and K pass through empty
    // asm statements at every call, so the compiler computes the addresses here instead of
    // keeping them in registers across the item loop.
    auto x_store = [&](int c0) {
        int ln = lane, Ko = K;
        asm volatile("" : "+v"(ln));
        asm volatile("" : "+s"(Ko));
#pragma unroll
        for (int r = 0; r < kRowsPerWave; ++r) {
            const int t = wave + NW * r;
            if constexpr (U::kTransposed) {
                bf16_t *xt = reinterpret_cast<bf16_t *>(Xs) + (t >> 5) * ((Ko + 1) * XP) + (t & 31);
#pragma unroll
                for (int m = 0; m < kXC; ++m) {
                    const int cb = c0 + 64 * m;
                    if (cb < Ko) xt[min(cb + ln, Ko) * XP] = bf16_t(v[r][m]);
                }
            } else {
                unsigned *dst = reinterpret_cast<unsigned *>(Xs) + t * XP + ln;
#pragma unroll
                for (int m = 0; m < kXC; ++m) {
                    unsigned w = v[r][m];
                    if constexpr (BF) w <<= 16;   // bf16 -> fp32, exact
                    const int cb = c0 + 64 * m;
                    if (cb + 64 <= Ko) dst[cb] = w;
                    else if (cb < Ko) dst[min(cb + ln, Ko) - ln] = w;
                }
            }
        }
    };
    auto item_tile = [&](int q, int64_t &t0_, int &rows_, int &s_) {
        const int tile = q / slices;
        s_ = q - tile * slices;
        t0_ = int64_t(tile) * TT;
        rows_ = int(T - t0_ < TT ? T - t0_ : TT);
    };
    int64_t t0;
    int rows, s;
    item_tile(q_first, t0, rows, s);
    x_load(t0, rows, 0, true);

    // Once: row pointers and bias to LDS (unplanned, wave 0 forms the unit row pointer).  A
    // pair's second product continues the first's unit row pointer (offset by the first's
    // units UA) and bias.
    [[maybe_unused]] int UA = 0;
    if constexpr (PAIR) {
        UA = uniform(clampi(uptr[NbA], 0, ucap));
        for (int i = threadIdx.x; i <= NbA; i += kThreads) s_up[i] = clampi(uptr[i], 0, ucap);
        for (int i = threadIdx.x; i < IB.Nb; i += kThreads)
            s_up[NbA + 1 + i] = UA + clampi(IB.uptr[i + 1], 0, IB.ucap);
        for (int i = threadIdx.x; i < NbA * R; i += kThreads) s_bias[i] = bias ? bias[i] : 0.0f;
        for (int i = threadIdx.x; i < IB.Nb * R; i += kThreads)
            s_bias[NbA * R + i] = IB.bias ? IB.bias[i] : 0.0f;
    } else if constexpr (PL) {
        for (int i = threadIdx.x; i <= Nb; i += kThreads) s_up[i] = clampi(uptr[i], 0, ucap);
    } else {
        for (int i = threadIdx.x; i <= Nb; i += kThreads) s_ib[i] = clampi(indptr[i], 0, nnzb);
    }
    if constexpr (!PAIR)
        for (int i = threadIdx.x; i < Nb * R; i += kThreads) s_bias[i] = bias ? bias[i] : 0.0f;
    __syncthreads();
    if constexpr (!PL) {
        if (wave == 0) {
            int carry = 0;
            for (int base = 0; base <= Nb; base += 64) {
                const int i = base + lane;
                const int n = i < Nb ? s_ib[i + 1] - s_ib[i] : 0;
                const int cnt = n > 0 ? (n + KB - 1) / KB : 0;
                const int incl = wave_scan_incl(cnt) + carry;
                if (i <= Nb) s_up[i] = incl - cnt;
                carry = __builtin_amdgcn_readlane(incl, 63);
            }
        }
        __syncthreads();
    }
    const int64_t k = uniform(s_up[Nb]);
    auto read_up_lds = [&](int i) { return uniform(s_up[i]); };
    auto read_ib_lds = [&](int i) { return uniform(s_ib[i]); };

    for (int q = q_first; q < q_end; q += nrank) {
        if (q != q_first) __syncthreads();   // the previous item's combine reads the X region

        // This item's X tile: chunks [0, kXC) are in registers; wider rows take more passes.
        x_store(0);
        for (int c0 = 64 * kXC; c0 < K; c0 += 64 * kXC) {
            x_load(t0, rows, c0, true);
            x_store(c0);
        }
        {
            int tid = int(threadIdx.x);
            asm volatile("" : "+v"(tid));
            if constexpr (U::kPad == 1) {   // the fp32 tile's zero pad column
                if (tid < TT) Xs[tid * XP + K] = 0.0f;
            }
            if constexpr (U::kTransposed) {   // the transposed tile's zero pad column K
                if (tid < TT)
                    reinterpret_cast<bf16_t *>(Xs)[(tid >> 5) * ((K + 1) * XP) + K * XP +
                                                   (tid & 31)] = 0;
            }
        }

        // The wave's share (as in the one-item kernel's LDS path).
        const int row_lo =
            (s == 0) ? 0 : uniform(wave_lower_bound(s_up, Nb, int64_t(s) * k / slices));
        const int row_hi = (s == slices - 1)
                               ? Nb
                               : uniform(wave_lower_bound(s_up, Nb, int64_t(s + 1) * k / slices));
        const int64_t Q0 = uniform(s_up[row_lo]);
        int64_t Q1 = uniform(s_up[row_hi]);
        if (Q1 < Q0) Q1 = Q0;
        static_assert(NW == 16, "wave starts are weighted for 16 waves");
        const unsigned span = unsigned(Q1 - Q0);
        const int ws = wave_start(Q0, span, unsigned(lane));
        const int wsn = wave_start(Q0, span, unsigned(lane) + 1);
        const int Pw = __builtin_amdgcn_readlane(ws, wave);
        const int Pw1 = __builtin_amdgcn_readlane(wsn, wave);
        int rlo = (wave == 0) ? row_lo : uniform(wave_lower_bound(s_up, Nb, int64_t(Pw)));
        rlo = rlo < row_lo ? row_lo : (rlo > row_hi ? row_hi : rlo);
        int rhi = (wave == NW - 1) ? row_hi : uniform(wave_lower_bound(s_up, Nb, int64_t(Pw1)));
        rhi = rhi < rlo ? rlo : (rhi > row_hi ? row_hi : rhi);
        int head_end = (rlo < rhi) ? uniform(s_up[rlo]) : Pw1;
        head_end = head_end < Pw ? Pw : (head_end > Pw1 ? Pw1 : head_end);
        int row = rlo - 1, end = head_end;
        if (head_end <= Pw) {
            end = 0;
            for (row = rlo; row < rhi; ++row) {
                const int p = uniform(s_up[row]);
                const int e = uniform(s_up[row + 1]);
                if (p < e) {
                    end = e < Pw1 ? e : Pw1;
                    break;
                }
            }
        }
        const bool has_head = head_end > Pw;

        // Prefetch cursor (unplanned): the row of the next unit to load, its units
        // [pr_u0, pr_u1) and blocks [pr_b0, pr_b1).
        int pr = row, pr_u0 = 0, pr_u1 = 0, pr_b0 = 0, pr_b1 = 0;
        auto fetch = [&](Ops &o, int &nvalid, int uu) {
            if constexpr (PAIR) {
                // Units from UA on are the second product's (its unit uu - UA); each range
                // ends at the wave's share, so past it nothing is read.
                const bool second = uu >= UA;
                const int32_t *cols = second ? IB.ucol : ucol;
                const void *vals = second ? IB.uval : uval;
                const int u2 = second ? uu - UA : uu;
                const int lim = second ? (Pw1 > UA ? Pw1 - UA : 0) : (Pw1 < UA ? Pw1 : UA);
                Src::load(o, u2, lim, cols, vals);
                nvalid = KB;
            } else if constexpr (PL) {
                Src::load(o, uu, Pw1, ucol, uval);
                nvalid = KB;
            } else {
                int p0 = nnzb, nv = KB;
                if (uu < Pw1) {
                    while (uu >= pr_u1 && pr < Nb - 1) {
                        ++pr;
                        pr_u0 = pr_u1;
                        pr_u1 = read_up_lds(pr + 1);
                        pr_b0 = read_ib_lds(pr);
                        pr_b1 = read_ib_lds(pr + 1);
                    }
                    p0 = pr_b0 + KB * (uu - pr_u0);
                    p0 = p0 < nnzb ? p0 : nnzb;
                    nv = pr_b1 - p0 < KB ? pr_b1 - p0 : KB;
                }
                U::load(o, p0, nnzb, indices, data);
                nvalid = nv;
            }
        };
        Ops ring[kRing];
        int nvr[kRing];
        if constexpr (!PL) {
            if (row < rhi) {
                pr_u0 = read_up_lds(row);
                pr_u1 = read_up_lds(row + 1);
                pr_b0 = read_ib_lds(row);
                pr_b1 = read_ib_lds(row + 1);
            }
        }
#pragma unroll
        for (int d = 0; d < kDepth; ++d) fetch(ring[d], nvr[d], Pw + d);
        __syncthreads();

        FlatItem fi{lane, wave, Pw, Pw1, rlo, rhi, row, end, has_head, ws, wsn, s_up, s_bias,
                    Xs, XP, Kb, reinterpret_cast<char *>(Xs) + I.wbuf_offset + wave * 2048,
                    TileOut{}, TileOut{}, PAIR ? NbA : INT_MAX};
        fi.out.ldy4 = int(ldy) * 4;
        fi.out.rsrc = buffer_rsrc(Y + t0 * ldy, unsigned(rows) * unsigned(fi.out.ldy4));
        if constexpr (PAIR) {
            fi.out2.ldy4 = int(IB.ldy) * 4;
            fi.out2.rsrc = buffer_rsrc(IB.Y + t0 * IB.ldy, unsigned(rows) * unsigned(fi.out2.ldy4));
        }

        // The next item's X rows, loaded under this item's stream.
        {
            const int qn = q + nrank;
            int64_t t0n = 0;
            int rowsn = 0, sn = 0;
            if (qn < q_end) item_tile(qn, t0n, rowsn, sn);
            x_load(t0n, rowsn, 0, false);
            t0 = t0n;
            rows = rowsn;
            s = sn;
        }
        flat_item_body<R, BF, PK, TT, PAIR>(fi, ring, nvr, fetch);
    }
}

template <int R, bool BF, int PK, int TT = 32>
bsr_status launch_flat_variant(const TiledBatch &batch, dim3 grid, size_t lds, bool persistent,
                               hipStream_t st, const LaunchEvents &ev, bool paired = false) {
    if constexpr (PK != 0) {
        if (paired) {
            launch_kernel(spmm_flat_persistent_kernel<R, BF, PK, TT, true>, grid,
                          dim3(kNW * 64), lds, st, ev, batch);
            return launch_status();
        }
    }
    if (persistent)
        launch_kernel(spmm_flat_persistent_kernel<R, BF, PK, TT>, grid, dim3(kNW * 64), lds, st,
                      ev, batch);
    else
        launch_kernel(spmm_flat_kernel<R, BF, PK, TT>, grid, dim3(kNW * 64), lds, st, ev, batch);
    return launch_status();
}

}  // namespace

bool flat_supported(int R, int C, int dtype) {
    return (dtype == BSR_F32 || dtype == BSR_BF16) && C == 1 && (R == 32 || R == 16);
}

int resolve_arith(int dtype, int arith) {
    if (arith == BSR_ARITH_AUTO) return BSR_ARITH_NATIVE;
    if (arith == BSR_ARITH_NATIVE || arith == BSR_ARITH_BF16X3) return arith;
    return -1;
}

bool plan_supported(int R, int C, int dtype, int arith) {
    const int a = resolve_arith(dtype, arith);
    if (a < 0 || (dtype != BSR_F32 && dtype != BSR_BF16) || C != 1 || R != 32) return false;
    return a == BSR_ARITH_NATIVE || dtype == BSR_F32;
}

int flat_unit_blocks(int R, int C, int dtype) {
    if (!flat_supported(R, C, dtype)) return 0;
    if (R == 32) return dtype == BSR_BF16 ? Unit<32, 1, true>::KB : Unit<32, 1, false>::KB;
    return Unit<16, 1, false>::KB;
}

bsr_status launch_spmm_flat(const TiledWork *work, int n, bool planned, void *stream,
                            const LaunchEvents &ev) {
    if (n < 1 || n > kMaxItems) return BSR_ERR_ARG;
    const int R = work[0].W->R, C = work[0].W->C;
    const bool bf = work[0].W->dtype == BSR_BF16;
    TiledBatch batch{};
    batch.n = n;
    int gx = 0;
    size_t lds = 0;
    for (int i = 0; i < n; ++i) {
        const TiledWork &w = work[i];
        if (w.W->R != R || w.W->C != C || w.W->dtype != work[0].W->dtype) return BSR_ERR_ARG;
        if ((w.plan_mem != nullptr) != planned) return BSR_ERR_ARG;
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
        if (planned) {
            const char *base = static_cast<const char *>(w.plan_mem);
            it.uptr = reinterpret_cast<const int32_t *>(base + w.plan_uptr_offset);
            it.ucol = reinterpret_cast<const int32_t *>(base + w.plan_col_offset);
            it.uval = base + w.plan_val_offset;
            it.ucap = int(w.plan_max_units);
        }
        it.partner = -1;
        const int wgs = ((w.plan.num_tiles * w.plan.slices + 7) / 8) * 8;
        if (wgs > gx) gx = wgs;
        if (w.plan.lds_bytes > lds) lds = w.plan.lds_bytes;
    }
    // More workgroups than CUs (one per CU fits): the persistent kernel, one workgroup per CU,
    // each walking several token tiles of its product.
    const int cus = device_cu_count() > 0 ? device_cu_count() : 256;
    // Paired products: a planned launch of an even number of products where products 2i and
    // 2i + 1 share X (same tensor, tokens, pitch and tile layout) and the persistent form is
    // taken runs n / 2 groups, each item covering one X tile of both products: the X store,
    // share computation and combine of an item are paid once for two products' work.  The LDS
    // head then holds both products' unit row pointers and biases.
    int pair_ipw[kMaxItems / 2] = {}, pair_bw[kMaxItems / 2] = {};
    size_t pair_lds = 0;
    bool paired = planned && n >= 2 && n % 2 == 0;
    for (int i = 0; paired && i + 1 < n; i += 2) {
        const TiledWork &a = work[i], &b = work[i + 1];
        paired = a.X == b.X && a.T == b.T && a.ldx == b.ldx && a.W->n_cols == b.W->n_cols &&
                 a.plan.x_pitch == b.plan.x_pitch && a.plan.num_tiles == b.plan.num_tiles &&
                 a.plan.slices == b.plan.slices && a.plan.tokens == b.plan.tokens &&
                 a.plan.wbuf_offset == b.plan.wbuf_offset && a.plan_arith == b.plan_arith;
        if (!paired) break;
        const int64_t nb2 = a.W->n_rows / R + b.W->n_rows / R;
        const int ipw = int((nb2 + 1 + 3) & ~int64_t(3)) + 4;   // + a spare word
        const int bw = int((a.W->n_rows + b.W->n_rows + 3) & ~int64_t(3));
        size_t rest = 0;   // the tile region (X tile, combine partials), as for one product
        for (const TiledWork *w : {&a, &b}) {
            const size_t r =
                w->plan.lds_bytes - size_t(w->plan.indptr_words + w->plan.bias_words) * 4;
            rest = r > rest ? r : rest;
        }
        const size_t need = size_t(ipw + bw) * 4 + rest;
        if (need > device_lds_per_block() || nb2 > INT_MAX / 64) paired = false;
        pair_ipw[i / 2] = ipw;
        pair_bw[i / 2] = bw;
        pair_lds = need > pair_lds ? need : pair_lds;
    }
    bool persistent = false;
    if (paired) {
        const int groups = n / 2;
        const int gp = (cus / groups) / 8 * 8;
        paired = int64_t(gx) * groups > cus && gp >= 8 && gp < gx;
        if (paired) {
            TiledBatch pb{};
            pb.n = n;
            for (int g = 0; g < groups; ++g) {
                pb.item[g] = batch.item[2 * g];
                pb.item[g].indptr_words = pair_ipw[g];
                pb.item[g].bias_words = pair_bw[g];
                pb.item[g].partner = groups + g;
                pb.item[groups + g] = batch.item[2 * g + 1];
            }
            batch = pb;
            gx = gp;
            lds = pair_lds;
            persistent = true;
        }
    }
    if (!paired && int64_t(gx) * n > cus) {
        const int gp = (cus / n) / 8 * 8;
        if (gp >= 8 && gp < gx) {
            gx = gp;
            persistent = true;
        }
    }
    hipStream_t st = as_stream(stream);
    const dim3 grid(gx, paired ? n / 2 : n);
    const bool split = planned && work[0].plan_arith == BSR_ARITH_BF16X3;
    const int tokens = work[0].plan.tokens;
    for (int i = 0; i < n; ++i) {
        if (planned && (work[i].plan_arith == BSR_ARITH_BF16X3) != split) return BSR_ERR_ARG;
        if (work[i].plan.tokens != tokens) return BSR_ERR_ARG;
    }
    if (tokens == 64 && !(R == 32 && bf)) return BSR_ERR_ARG;
    if (R == 32) {
        if (bf) {
            if (split) return BSR_ERR_UNSUPPORTED;
            if (tokens == 64)
                return planned ? launch_flat_variant<32, true, 1, 64>(batch, grid, lds,
                                                                      persistent, st, ev, paired)
                               : launch_flat_variant<32, true, 0, 64>(batch, grid, lds,
                                                                      persistent, st, ev);
            return planned
                       ? launch_flat_variant<32, true, 1>(batch, grid, lds, persistent, st, ev,
                                                          paired)
                       : launch_flat_variant<32, true, 0>(batch, grid, lds, persistent, st, ev);
        }
        if (split)
            return launch_flat_variant<32, false, 2>(batch, grid, lds, persistent, st, ev, paired);
        return planned
                   ? launch_flat_variant<32, false, 1>(batch, grid, lds, persistent, st, ev, paired)
                   : launch_flat_variant<32, false, 0>(batch, grid, lds, persistent, st, ev);
    }
    if (planned) return BSR_ERR_UNSUPPORTED;
    if (bf) return launch_flat_variant<16, true, 0>(batch, grid, lds, persistent, st, ev);
    return launch_flat_variant<16, false, 0>(batch, grid, lds, persistent, st, ev);
}

}  // namespace bsr
