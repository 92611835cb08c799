// Attention weights P = softmax(S + M) written K-major with their token
// energies (Sec. 3.3: the token scores of the value product are the column
// norms of P; the Limitations section names the memory movement of a
// separate scoring pass as a cost to remove).
//
//   rmax[i]   = max over kept t of S[i][t],  rsum[i] = sum over kept t of
//               exp(S[i][t] - rmax[i])                         (fp32)
//   Pt[t][i]  = bf16(exp(S[i][t] - rmax[i]) / rsum[i]), 0 where masked
//   energy[t] = sum over i of Pt[t][i]^2                       (float64)
//
// Two launches, as for the normalisation producer.  softmax_rowstats_kernel:
// one wave per query row reads the row's kept scores once (with the causal
// mask, only the keys up to the row's limit: the masked half of S is never
// read), keeping a running maximum and a sum rescaled whenever the maximum
// rises, per lane in key order and then merged across the wave in a fixed
// butterfly (every lane ends with the same pair).  Then the scoring pass's
// transposing tile kernel in its softmax variant forms the weights in
// registers and writes them K-major as whole 128-byte row segments with the
// float64 column energies; its wave tiles that lie wholly above the causal
// diagonal read nothing and write zeros.
#include <cmath>

#include "device_common.h"
#include "kernels.h"

namespace rmm {

namespace {

constexpr int kRowThreads = 256;   // four rows per workgroup, one per wave

__device__ __forceinline__ void merge_stats(float &m, float &l, float m2, float l2) {
    const float mm = fmaxf(m, m2);
    if (mm == -INFINITY) return;                 // both empty
    const float a = m == -INFINITY ? 0.f : l * __expf(m - mm);
    const float b = m2 == -INFINITY ? 0.f : l2 * __expf(m2 - mm);
    m = mm;
    l = a + b;
}

__global__ __launch_bounds__(kRowThreads) void softmax_rowstats_kernel(
    const uint16_t *__restrict__ S, int64_t U, int64_t Lq, int64_t Lk, int64_t lds, int causal,
    float *__restrict__ rmax, float *__restrict__ rinv) {
    const int lane = threadIdx.x & 63;
    const int64_t row = static_cast<int64_t>(blockIdx.x) * (kRowThreads / 64) + (threadIdx.x >> 6);
    if (row >= U * Lq) return;                   // whole waves leave together
    const int64_t i = row % Lq;
    const uint16_t *s = S + row * lds;           // units are packed: unit stride Lq * lds
    // keys 0 .. nk-1 are kept (the causal mask keeps t <= i + Lk - Lq)
    const int64_t nk = causal ? max<int64_t>(0, min<int64_t>(Lk, i + Lk - Lq + 1)) : Lk;
    const int64_t nc = (nk + 7) / 8;
    float m = -INFINITY, l = 0.f;
    for (int64_t c0 = lane; c0 < nc; c0 += 4 * 64) {
        uint4 q[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int64_t c = c0 + 64 * u;
            q[u] = c < nc ? *reinterpret_cast<const uint4 *>(s + 8 * c) : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int64_t c = c0 + 64 * u;
            if (c >= nc) break;
            const uint32_t w[4] = {q[u].x, q[u].y, q[u].z, q[u].w};
            float v[8];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                v[2 * e] = __uint_as_float(w[e] << 16);
                v[2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u);
            }
            float cm = -INFINITY;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                if (8 * c + e >= nk) v[e] = -INFINITY;
                cm = fmaxf(cm, v[e]);
            }
            if (cm == -INFINITY) continue;         // every key of the chunk masked
            if (cm > m) {
                l = m == -INFINITY ? 0.f : l * __expf(m - cm);
                m = cm;
            }
#pragma unroll
            for (int e = 0; e < 8; ++e) l += __expf(v[e] - m);   // exp(-inf) = 0
        }
    }
#pragma unroll
    for (int sh = 1; sh < 64; sh <<= 1) {
        const float m2 = __shfl_xor(m, sh), l2 = __shfl_xor(l, sh);
        merge_stats(m, l, m2, l2);
    }
    if (lane == 0) {
        const bool empty = !(l > 0.f);
        rmax[row] = empty ? 0.f : m;
        rinv[row] = empty ? 0.f : 1.0f / l;
    }
}

inline size_t align256(size_t n) { return (n + 255) & ~static_cast<size_t>(255); }

}  // namespace

size_t weights_workspace_bytes(int64_t U, int64_t Lq, int64_t Lk) {
    return 2 * align256(static_cast<size_t>(U * Lq) * sizeof(float)) + score_workspace_bytes(U, Lq, Lk);
}

hipError_t launch_attention_weights_kmajor(const uint16_t *S, int64_t U, int64_t Lq, int64_t Lk,
                                           int64_t lds, int causal, const float *rmax_in,
                                           const float *rinv_in, uint16_t *Pt, int64_t ldpt,
                                           double *energy, void *workspace, hipStream_t stream) {
    char *ws = static_cast<char *>(workspace);
    float *rmax = reinterpret_cast<float *>(ws);
    float *rinv = reinterpret_cast<float *>(ws + align256(static_cast<size_t>(U * Lq) * sizeof(float)));
    double *partials = reinterpret_cast<double *>(ws + 2 * align256(static_cast<size_t>(U * Lq) * sizeof(float)));
    if (rmax_in && rinv_in)
        return launch_score_softmax_kmajor(S, U, Lq, Lk, lds, rmax_in, rinv_in, Lk - Lq, causal, energy,
                                           partials, Pt, ldpt, stream);
    const int64_t rows = U * Lq, per = kRowThreads / 64;
    hipLaunchKernelGGL(softmax_rowstats_kernel, dim3(static_cast<unsigned>((rows + per - 1) / per)),
                       dim3(kRowThreads), 0, stream, S, U, Lq, Lk, lds, causal, rmax, rinv);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_score_softmax_kmajor(S, U, Lq, Lk, lds, rmax, rinv, Lk - Lq, causal, energy, partials,
                                       Pt, ldpt, stream);
}

}  // namespace rmm
