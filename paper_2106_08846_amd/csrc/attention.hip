// Scaled dot-product attention of the BERT attention block whose projections are the pruned
// BSR products (Sec. 2.3 prunes BERT's attention weights; Table 1 times the whole model):
//
//   ctx[b, s, head h] = sum_j softmax_j(scale * <Q[b,s,h], K[b,j,h]>) V[b,j,h]
//
// Tokens are rows t = b * seq + s of Q, K, V and ctx; head h owns columns h*64 .. h*64 + 63.
// No mask: every token attends to every token of its sequence.  fp32 throughout.
//
// One workgroup of 8 * QT threads computes QT queries (32, or 8 when 32-query tiles would not
// give every CU a workgroup) of one (sequence, head).  The keys are
// visited in blocks of 64: the block's K and V rows are staged in LDS (row pitch 68 floats, so
// rows start 4 banks apart and the 16-byte reads below are conflict-free), and the softmax is
// kept online (running maximum m, running sum l, output rescaled by exp(m_old - m_new)), so no
// score matrix is stored.  Thread t serves query t / 8; its 8 lanes split the block's keys for
// the scores (lane u takes keys u, u + 8, ...) and the 64 output columns for P V (lane u takes
// columns 8u .. 8u + 7); the row's maximum and sum are combined across the 8 lanes with xor
// shuffles, and the row's weights pass from the score lanes to the output lanes through LDS.
#include <cmath>

#include "device_common.h"

namespace bsr {

namespace {

constexpr int kKB = 64;       // keys per block
constexpr int kD = 64;        // head width
constexpr int kPitch = 68;    // LDS row pitch, floats
constexpr int kMfmaMinSeq = 128;   // shortest sequence for the matrix-core kernel
constexpr int kSplitBelow = 2;     // key-split 8-query tiles below this many tiles per CU

typedef float floatx4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ floatx4 load4(const float *p) {
    return *reinterpret_cast<const floatx4 *>(p);
}

__device__ __forceinline__ float row_max8(float x) {
    x = fmaxf(x, __shfl_xor(x, 1));
    x = fmaxf(x, __shfl_xor(x, 2));
    return fmaxf(x, __shfl_xor(x, 4));
}

__device__ __forceinline__ float row_sum8(float x) {
    x += __shfl_xor(x, 1);
    x += __shfl_xor(x, 2);
    return x + __shfl_xor(x, 4);
}

template <int kQT>
__global__ __launch_bounds__(kQT * 8) void attention_kernel(
    const float *__restrict__ Q, int64_t ldq, const float *__restrict__ K, int64_t ldk,
    const float *__restrict__ V, int64_t ldv, float *__restrict__ O, int64_t ldo, int seq,
    float scale) {
    constexpr int kThreads = kQT * 8;
    __shared__ float Ks[kKB * kPitch];
    __shared__ float Vs[kKB * kPitch];
    __shared__ float Ps[kQT * kPitch];
    const int tid = threadIdx.x, qi = tid >> 3, u = tid & 7;
    const int q0 = blockIdx.x * kQT, h = blockIdx.y;
    const int64_t tok0 = int64_t(blockIdx.z) * seq;
    const int qrow = q0 + qi;
    const bool qvalid = qrow < seq;

    // This thread's query row, pre-scaled (rows past the sequence read row 0; never stored).
    float q[kD];
    {
        const float *qp = Q + (tok0 + (qvalid ? qrow : 0)) * ldq + h * kD;
#pragma unroll
        for (int d = 0; d < kD; d += 4) {
            const floatx4 v = load4(qp + d);
#pragma unroll
            for (int e = 0; e < 4; ++e) q[d + e] = v[e] * scale;
        }
    }
    float m = -INFINITY, l = 0.0f, acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.0f;

    for (int k0 = 0; k0 < seq; k0 += kKB) {
        __syncthreads();   // the previous block's LDS reads are done
        // Stage K and V rows k0 .. k0 + 63 of this head (rows past the sequence are zero).
        // Four 16-byte pieces of K and of V per thread in flight, then their LDS stores.
        constexpr int kPer = kKB * (kD / 4) / kThreads;   // pieces per thread
        constexpr int kBatch = kPer < 4 ? kPer : 4;
#pragma unroll
        for (int n0 = 0; n0 < kPer; n0 += kBatch) {
            floatx4 kst[kBatch], vst[kBatch];
#pragma unroll
            for (int n = 0; n < kBatch; ++n) {
                const int i = tid + (n0 + n) * kThreads;
                const int r = i >> 4, c4 = (i & 15) * 4;
                const int key = k0 + r < seq ? k0 + r : seq - 1;   // past the end: zeroed below
                kst[n] = load4(K + (tok0 + key) * ldk + h * kD + c4);
                vst[n] = load4(V + (tok0 + key) * ldv + h * kD + c4);
            }
#pragma unroll
            for (int n = 0; n < kBatch; ++n) {
                const int i = tid + (n0 + n) * kThreads;
                const int r = i >> 4, c4 = (i & 15) * 4;
                const floatx4 z = {0.0f, 0.0f, 0.0f, 0.0f};
                *reinterpret_cast<floatx4 *>(&Ks[r * kPitch + c4]) = k0 + r < seq ? kst[n] : z;
                *reinterpret_cast<floatx4 *>(&Vs[r * kPitch + c4]) = k0 + r < seq ? vst[n] : z;
            }
        }
        __syncthreads();

        // Scores of keys u + 8j (j < 8), the eight dot products advanced together (eight
        // independent FMA chains); keys past the sequence get -inf (weight 0).
        float s[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) s[j] = 0.0f;
#pragma unroll
        for (int d = 0; d < kD; d += 4) {
            floatx4 kv[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) kv[j] = load4(&Ks[(u + 8 * j) * kPitch + d]);
#pragma unroll
            for (int e = 0; e < 4; ++e)
#pragma unroll
                for (int j = 0; j < 8; ++j) s[j] = __builtin_fmaf(q[d + e], kv[j][e], s[j]);
        }
#pragma unroll
        for (int j = 0; j < 8; ++j)
            if (k0 + u + 8 * j >= seq) s[j] = -INFINITY;
        float bm = s[0];
#pragma unroll
        for (int j = 1; j < 8; ++j) bm = fmaxf(bm, s[j]);
        const float mn = fmaxf(m, row_max8(bm));   // finite: key k0 exists
        const float corr = expf(m - mn);           // 0 on the first block (m = -inf)
        float ps = 0.0f;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const float p = expf(s[j] - mn);
            ps += p;
            Ps[qi * kPitch + u + 8 * j] = p;
        }
        l = l * corr + row_sum8(ps);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] *= corr;
        m = mn;
        __syncthreads();   // the row's weights are in LDS

        const float *pr = &Ps[qi * kPitch];
#pragma unroll 8
        for (int r = 0; r < kKB; ++r) {
            const float p = pr[r];
            const floatx4 v0 = load4(&Vs[r * kPitch + 8 * u]);
            const floatx4 v1 = load4(&Vs[r * kPitch + 8 * u + 4]);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                acc[e] = __builtin_fmaf(p, v0[e], acc[e]);
                acc[4 + e] = __builtin_fmaf(p, v1[e], acc[4 + e]);
            }
        }
    }
    if (qvalid) {
        float *op = O + (tok0 + qrow) * ldo + h * kD + 8 * u;
#pragma unroll
        for (int e = 0; e < 8; ++e) op[e] = acc[e] / l;
    }
}

// Short sequences with few (sequence, head) pairs: kKS groups of 8 queries x 8 lanes (one wave
// each) serve the same queries; group ks takes the key blocks ks, ks + kKS, ... with the online
// softmax above, and the groups' partial results are merged at the end.  Each group has its own
// K, V and P buffers in (dynamic) LDS.
template <int kKS>
__global__ __launch_bounds__(64 * kKS) void attention_split_kernel(
    const float *__restrict__ Q, int64_t ldq, const float *__restrict__ K, int64_t ldk,
    const float *__restrict__ V, int64_t ldv, float *__restrict__ O, int64_t ldo, int seq,
    float scale) {
    constexpr int kQT = 8;
    constexpr int kThreads = kQT * 8;             // threads per group
    constexpr int kGroupFloats = 2 * kKB * kPitch + kQT * kPitch;
    extern __shared__ float smem[];
    const int ks = threadIdx.x / kThreads, tid = threadIdx.x % kThreads;
    float *Ks = smem + ks * kGroupFloats;
    float *Vs = Ks + kKB * kPitch;
    float *Ps = Vs + kKB * kPitch;
    const int qi = tid >> 3, u = tid & 7;
    const int q0 = blockIdx.x * kQT, h = blockIdx.y;
    const int64_t tok0 = int64_t(blockIdx.z) * seq;
    const int qrow = q0 + qi;
    const bool qvalid = qrow < seq;

    // This thread's query row, pre-scaled (rows past the sequence read row 0; never stored).
    float q[kD];
    {
        const float *qp = Q + (tok0 + (qvalid ? qrow : 0)) * ldq + h * kD;
#pragma unroll
        for (int d = 0; d < kD; d += 4) {
            const floatx4 v = load4(qp + d);
#pragma unroll
            for (int e = 0; e < 4; ++e) q[d + e] = v[e] * scale;
        }
    }
    float m = -INFINITY, l = 0.0f, acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.0f;

    // Every group runs the same number of rounds (and barriers); a group whose block is past
    // the end of the sequence idles through its round.
    const int nblk = (seq + kKB - 1) / kKB;
    const int rounds = (nblk + kKS - 1) / kKS;
    for (int it = 0; it < rounds; ++it) {
        const int k0 = (ks + kKS * it) * kKB;
        const bool active = k0 < seq;
        __syncthreads();   // the previous block's LDS reads are done
        // Stage K and V rows k0 .. k0 + 63 of this head (rows past the sequence are zero).
        // Four 16-byte pieces of K and of V per thread in flight, then their LDS stores.
        constexpr int kPer = kKB * (kD / 4) / kThreads;   // pieces per thread
        constexpr int kBatch = kPer < 4 ? kPer : 4;
        if (active) {
#pragma unroll
            for (int n0 = 0; n0 < kPer; n0 += kBatch) {
                floatx4 kst[kBatch], vst[kBatch];
#pragma unroll
                for (int n = 0; n < kBatch; ++n) {
                    const int i = tid + (n0 + n) * kThreads;
                    const int r = i >> 4, c4 = (i & 15) * 4;
                    const int key = k0 + r < seq ? k0 + r : seq - 1;   // past the end: zeroed
                    kst[n] = load4(K + (tok0 + key) * ldk + h * kD + c4);
                    vst[n] = load4(V + (tok0 + key) * ldv + h * kD + c4);
                }
#pragma unroll
                for (int n = 0; n < kBatch; ++n) {
                    const int i = tid + (n0 + n) * kThreads;
                    const int r = i >> 4, c4 = (i & 15) * 4;
                    const floatx4 z = {0.0f, 0.0f, 0.0f, 0.0f};
                    *reinterpret_cast<floatx4 *>(&Ks[r * kPitch + c4]) = k0 + r < seq ? kst[n] : z;
                    *reinterpret_cast<floatx4 *>(&Vs[r * kPitch + c4]) = k0 + r < seq ? vst[n] : z;
                }
            }
        }
        __syncthreads();

        if (active) {
            // Scores of keys u + 8j (j < 8), the eight dot products advanced together (eight
            // independent FMA chains); keys past the sequence get -inf (weight 0).
            float s[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) s[j] = 0.0f;
#pragma unroll
            for (int d = 0; d < kD; d += 4) {
                floatx4 kv[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) kv[j] = load4(&Ks[(u + 8 * j) * kPitch + d]);
#pragma unroll
                for (int e = 0; e < 4; ++e)
#pragma unroll
                    for (int j = 0; j < 8; ++j) s[j] = __builtin_fmaf(q[d + e], kv[j][e], s[j]);
            }
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if (k0 + u + 8 * j >= seq) s[j] = -INFINITY;
            float bm = s[0];
#pragma unroll
            for (int j = 1; j < 8; ++j) bm = fmaxf(bm, s[j]);
            const float mn = fmaxf(m, row_max8(bm));   // finite: key k0 exists
            const float corr = expf(m - mn);           // 0 on the group's first block
            float ps = 0.0f;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const float p = expf(s[j] - mn);
                ps += p;
                Ps[qi * kPitch + u + 8 * j] = p;
            }
            l = l * corr + row_sum8(ps);
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[e] *= corr;
            m = mn;
        }
        __syncthreads();   // the row's weights are in LDS

        if (active) {
            const float *pr = &Ps[qi * kPitch];
#pragma unroll 8
            for (int r = 0; r < kKB; ++r) {
                const float p = pr[r];
                const floatx4 v0 = load4(&Vs[r * kPitch + 8 * u]);
                const floatx4 v1 = load4(&Vs[r * kPitch + 8 * u + 4]);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    acc[e] = __builtin_fmaf(p, v0[e], acc[e]);
                    acc[4 + e] = __builtin_fmaf(p, v1[e], acc[4 + e]);
                }
            }
        }
    }
    {
        // Merge the groups in group order: with M the largest running maximum,
        // out = sum_g acc_g exp(m_g - M) / sum_g l_g exp(m_g - M).  A group that saw no key
        // has m = -inf, l = 0 and adds nothing; group 0 always saw key 0.
        constexpr int kSlot = 8 * 8 + 2;   // per thread: acc, then m and l
        __syncthreads();
        float *C = smem + (ks * kThreads + tid) * kSlot;
#pragma unroll
        for (int e = 0; e < 8; ++e) C[e] = acc[e];
        C[64] = m;
        C[65] = l;
        __syncthreads();
        if (ks != 0) return;
        float M = m;
#pragma unroll
        for (int g = 1; g < kKS; ++g) M = fmaxf(M, smem[(g * kThreads + tid) * kSlot + 64]);
        const float w0 = expf(m - M);
        l *= w0;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] *= w0;
#pragma unroll
        for (int g = 1; g < kKS; ++g) {
            const float *Cg = smem + (g * kThreads + tid) * kSlot;
            const float w = expf(Cg[64] - M);   // 0 for a group without keys
            l = __builtin_fmaf(Cg[65], w, l);
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[e] = __builtin_fmaf(Cg[e], w, acc[e]);
        }
    }
    if (qvalid) {
        float *op = O + (tok0 + qrow) * ldo + h * kD + 8 * u;
#pragma unroll
        for (int e = 0; e < 8; ++e) op[e] = acc[e] / l;
    }
}

// ------------------------------------------------------------------- matrix-core version
// One wave computes 32 queries of one (sequence, head) on v_mfma_f32_32x32x2_f32; kWQ waves of
// a workgroup share the staged keys and values (blocks of 64, as above).  Lane l serves query
// l % 32 as half hh = l / 32.
//   Scores, transposed: S^T = K Q^T for each group of 32 keys.  Step s (s < 32) contracts
//   dimension s + 32hh in slot hh: A = K[key l%32][s + 32hh] (LDS), B = the lane's pre-scaled
//   q[s + 32hh] (registers).  Register v of lane l then holds the score of query l % 32 and
//   key 8(v/4) + 4hh + v%4 of the group, so a query's 32 scores sit in the lane pair
//   (l, l ^ 32): the group maximum and sum take 15 register operations and one exchange.
//   Output, transposed: O^T += V^T P^T.  Step v contracts the two keys that register v holds in
//   the two halves: A = V[that key][32t + l%32] (LDS; output column tile t = 0, 1), B = this
//   lane's weight p[v], so the weights never leave their registers.
// The online softmax is the one above (running maximum and sum per query, output rescaled by
// exp(m_old - m_new)); each query's running values are kept, identical, in both its lanes.
template <int kWQ, int kKS>
__global__ __launch_bounds__(kWQ * kKS * 64) __attribute__((amdgpu_waves_per_eu(3)))
void attention_mfma_kernel(
    const float *__restrict__ Q, int64_t ldq, const float *__restrict__ K, int64_t ldk,
    const float *__restrict__ V, int64_t ldv, float *__restrict__ O, int64_t ldo, int seq,
    float scale) {
    // kKS = 2: two waves serve each query tile, one taking the first 32 keys of every staged
    // block and the other the second 32, and merge their results at the end.
    static_assert(kKS == 1 || kKS == 2, "one or two waves per query tile");
    typedef float floatx16 __attribute__((ext_vector_type(16)));
    constexpr int kThreads = kWQ * kKS * 64;
    __shared__ float Ks[kKB * kPitch];
    __shared__ float Vs[kKB * kPitch];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int qw = wave % kWQ, ks = wave / kWQ;
    const int ql = lane & 31, hh = lane >> 5;
    const int qrow = (blockIdx.x * kWQ + qw) * 32 + ql, h = blockIdx.y;
    const int64_t tok0 = int64_t(blockIdx.z) * seq;
    const bool qvalid = qrow < seq;

    // Half hh of this lane's query row, pre-scaled (rows past the sequence read row 0; never
    // stored).
    float q[32];
    {
        const float *qp = Q + (tok0 + (qvalid ? qrow : 0)) * ldq + h * kD + 32 * hh;
#pragma unroll
        for (int d = 0; d < 32; d += 4) {
            const floatx4 v = load4(qp + d);
#pragma unroll
            for (int e = 0; e < 4; ++e) q[d + e] = v[e] * scale;
        }
    }
    float m = -INFINITY, l = 0.0f;
    floatx16 o0, o1;
#pragma unroll
    for (int v = 0; v < 16; ++v) o0[v] = o1[v] = 0.0f;

    for (int k0 = 0; k0 < seq; k0 += kKB) {
        __syncthreads();   // the previous block's LDS reads are done
        // Stage K and V rows k0 .. k0 + 63 of this head (rows past the sequence are zero).
        constexpr int kPer = kKB * (kD / 4) / kThreads;   // 16-byte pieces per thread
        constexpr int kBatch = kPer < 4 ? kPer : 4;
#pragma unroll
        for (int n0 = 0; n0 < kPer; n0 += kBatch) {
            floatx4 kst[kBatch], vst[kBatch];
#pragma unroll
            for (int n = 0; n < kBatch; ++n) {
                const int i = tid + (n0 + n) * kThreads;
                const int r = i >> 4, c4 = (i & 15) * 4;
                const int key = k0 + r < seq ? k0 + r : seq - 1;   // past the end: zeroed below
                kst[n] = load4(K + (tok0 + key) * ldk + h * kD + c4);
                vst[n] = load4(V + (tok0 + key) * ldv + h * kD + c4);
            }
#pragma unroll
            for (int n = 0; n < kBatch; ++n) {
                const int i = tid + (n0 + n) * kThreads;
                const int r = i >> 4, c4 = (i & 15) * 4;
                const floatx4 z = {0.0f, 0.0f, 0.0f, 0.0f};
                *reinterpret_cast<floatx4 *>(&Ks[r * kPitch + c4]) = k0 + r < seq ? kst[n] : z;
                *reinterpret_cast<floatx4 *>(&Vs[r * kPitch + c4]) = k0 + r < seq ? vst[n] : z;
            }
        }
        __syncthreads();

#pragma unroll
        for (int gi = 0; gi < kKB / 32 / kKS; ++gi) {
            const int g = gi * kKS + ks;
            const int kg = k0 + 32 * g;
            if (kg >= seq) break;   // the whole group is past the end
            floatx16 s;
#pragma unroll
            for (int v = 0; v < 16; ++v) s[v] = 0.0f;
            const float *kr = &Ks[(32 * g + ql) * kPitch + 32 * hh];
#pragma unroll
            for (int d = 0; d < 32; d += 4) {
                const floatx4 kv = load4(kr + d);
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    s = __builtin_amdgcn_mfma_f32_32x32x2f32(kv[e], q[d + e], s, 0, 0, 0);
            }
            // Keys past the sequence get -inf (weight 0); the group's first key exists.
            float mx = -INFINITY;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int key = kg + 8 * (v >> 2) + 4 * hh + (v & 3);
                if (key >= seq) s[v] = -INFINITY;
                mx = fmaxf(mx, s[v]);
            }
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            const float mn = fmaxf(m, mx);
            const float corr = expf(m - mn);   // 0 on the first group (m = -inf)
            float ps = 0.0f;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                s[v] = expf(s[v] - mn);
                ps += s[v];
            }
            ps += __shfl_xor(ps, 32);
            l = l * corr + ps;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                o0[v] *= corr;
                o1[v] *= corr;
            }
            m = mn;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const float *vr = &Vs[(32 * g + 8 * (v >> 2) + 4 * hh + (v & 3)) * kPitch + ql];
                o0 = __builtin_amdgcn_mfma_f32_32x32x2f32(vr[0], s[v], o0, 0, 0, 0);
                o1 = __builtin_amdgcn_mfma_f32_32x32x2f32(vr[32], s[v], o1, 0, 0, 0);
            }
        }
    }
    if constexpr (kKS == 2) {
        // Merge the two key halves: the second wave of each tile leaves its running maximum,
        // sum and output in LDS (the K buffer is free after the barrier); the first adds
        // them, both rescaled to the larger maximum.  A wave that saw no key (sequences of at
        // most 32) has m = -inf, l = 0 and adds nothing.
        constexpr int kSlot = 34;   // floats per lane: o0, o1, m, l
        static_assert(kWQ * 64 * kSlot <= kKB * kPitch, "merge buffer fits in the K buffer");
        __syncthreads();
        float *C = Ks + (qw * 64 + lane) * kSlot;
        if (ks == 1) {
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                C[v] = o0[v];
                C[16 + v] = o1[v];
            }
            C[32] = m;
            C[33] = l;
        }
        __syncthreads();
        if (ks == 1) return;
        const float m1 = C[32], M = fmaxf(m, m1);
        const float w0 = expf(m - M), w1 = expf(m1 - M);
        l = l * w0 + C[33] * w1;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            o0[v] = o0[v] * w0 + C[v] * w1;
            o1[v] = o1[v] * w0 + C[16 + v] * w1;
        }
    }
    // Register v of tile t holds O[query][32t + 8(v/4) + 4hh + v%4]: four consecutive columns
    // per group of four registers, stored as 16 bytes.
    if (qvalid) {
        float *op = O + (tok0 + qrow) * ldo + h * kD + 4 * hh;
#pragma unroll
        for (int v4 = 0; v4 < 4; ++v4) {
            floatx4 a, b;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                a[e] = o0[4 * v4 + e] / l;
                b[e] = o1[4 * v4 + e] / l;
            }
            *reinterpret_cast<floatx4 *>(op + 8 * v4) = a;
            *reinterpret_cast<floatx4 *>(op + 32 + 8 * v4) = b;
        }
    }
}

}  // namespace

bsr_status launch_attention(const float *Q, int64_t ldq, const float *K, int64_t ldk,
                            const float *V, int64_t ldv, float *O, int64_t ldo, int batch,
                            int seq, int heads, float scale, void *stream) {
    const int64_t tiles32 = int64_t((seq + 31) / 32) * heads * batch;
    const int cus = device_cu_count() > 0 ? device_cu_count() : 256;
    // The matrix-core kernel for sequences of 2 * kMfmaMinSeq keys or more, and for sequences
    // of kMfmaMinSeq keys or more when there are at least three 32-query tiles per CU (its
    // per-wave chain of key groups is long; measured on MI355X, shorter sequences with fewer
    // tiles run faster on the vector ALUs).  Up to eight tiles per CU, two waves split each tile's keys (twice the
    // waves); beyond that, four tiles share each workgroup's staged keys.
    if (seq >= 2 * kMfmaMinSeq || (seq >= kMfmaMinSeq && tiles32 >= 3 * int64_t(cus))) {
        if (tiles32 >= 8 * int64_t(cus)) {
            const dim3 grid(unsigned((seq + 127) / 128), unsigned(heads), unsigned(batch));
            hipLaunchKernelGGL((attention_mfma_kernel<4, 1>), grid, dim3(256), 0,
                               as_stream(stream), Q, ldq, K, ldk, V, ldv, O, ldo, seq, scale);
        } else {
            const dim3 grid(unsigned((seq + 63) / 64), unsigned(heads), unsigned(batch));
            hipLaunchKernelGGL((attention_mfma_kernel<2, 2>), grid, dim3(256), 0,
                               as_stream(stream), Q, ldq, K, ldk, V, ldv, O, ldo, seq, scale);
        }
        return launch_status();
    }
    // Vector-ALU kernels: 32-query tiles when they give at least one workgroup per CU, else
    // 8-query tiles; when even those give fewer than kSplitBelow waves per CU, two or four
    // waves split the keys of each tile.
    const int nblk = (seq + kKB - 1) / kKB;
    const int64_t tiles8 = int64_t((seq + 7) / 8) * heads * batch;
    if (tiles32 >= cus) {
        const dim3 grid(unsigned((seq + 31) / 32), unsigned(heads), unsigned(batch));
        hipLaunchKernelGGL(attention_kernel<32>, grid, dim3(256), 0, as_stream(stream), Q, ldq, K,
                           ldk, V, ldv, O, ldo, seq, scale);
        return launch_status();
    }
    const dim3 grid(unsigned((seq + 7) / 8), unsigned(heads), unsigned(batch));
    const int ks = tiles8 >= kSplitBelow * int64_t(cus) || nblk < 2 ? 1 : (nblk < 4 ? 2 : 4);
    const size_t lds = size_t(ks) * (2 * kKB * kPitch + 8 * kPitch) * sizeof(float);
    if (ks == 1)
        hipLaunchKernelGGL(attention_kernel<8>, grid, dim3(64), 0, as_stream(stream), Q, ldq, K,
                           ldk, V, ldv, O, ldo, seq, scale);
    else if (ks == 2)
        hipLaunchKernelGGL(attention_split_kernel<2>, grid, dim3(128), lds, as_stream(stream), Q,
                           ldq, K, ldk, V, ldv, O, ldo, seq, scale);
    else
        hipLaunchKernelGGL(attention_split_kernel<4>, grid, dim3(256), lds, as_stream(stream), Q,
                           ldq, K, ldk, V, ldv, O, ldo, seq, scale);
    return launch_status();
}

}  // namespace bsr
