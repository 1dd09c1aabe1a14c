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

}  // namespace

bsr_status launch_attention(const float *Q, int64_t ldq, const float *K, int64_t ldk,
                            const float *V, int64_t ldv, float *O, int64_t ldo, int batch,
                            int seq, int heads, float scale, void *stream) {
    // 32-query tiles when they give at least one workgroup per CU, else 8-query tiles.
    const int64_t tiles32 = int64_t((seq + 31) / 32) * heads * batch;
    const int cus = device_cu_count() > 0 ? device_cu_count() : 256;
    if (tiles32 >= cus) {
        const dim3 grid(unsigned((seq + 31) / 32), unsigned(heads), unsigned(batch));
        hipLaunchKernelGGL(attention_kernel<32>, grid, dim3(256), 0, as_stream(stream), Q, ldq, K,
                           ldk, V, ldv, O, ldo, seq, scale);
    } else {
        const dim3 grid(unsigned((seq + 7) / 8), unsigned(heads), unsigned(batch));
        hipLaunchKernelGGL(attention_kernel<8>, grid, dim3(64), 0, as_stream(stream), Q, ldq, K,
                           ldk, V, ldv, O, ldo, seq, scale);
    }
    return launch_status();
}

}  // namespace bsr
