// Reduced attention scores over head-dim slices (Sec. 3.3, Attention):
//   S[h] = scale * Q[h][:, I_h] K[g(h)][:, I_h]^T,  -inf where causally masked,
// with g(h) = h / (H / Hkv).
//
// Both operands are rows gathered along the head dimension (a Q row and a K
// row are each D contiguous values), so each k-tile is a lane-along-t gather
// into n-major / m-major LDS tiles that feed v_mfma_f32_32x32x16_bf16
// directly.  The kernel is bound by writing S (Lq*Lk values per head), which
// does not shrink with k; tiles lying wholly above the causal diagonal skip
// the product and only write -inf.
#include "device_common.h"
#include "kernels.h"

namespace rmm {

namespace {

constexpr uint16_t kBf16NegInf = 0xff80;

template <int BM, int BN, int BK, int WM, int WN>
__global__ __launch_bounds__(WM *WN *kWave) void qk_bf16_kernel(
    const uint16_t *__restrict__ Q, const uint16_t *__restrict__ Kc,
    const int32_t *__restrict__ idx, uint16_t *__restrict__ S, int H, int Hkv, int Lq, int Lk,
    int D, int k, float scale, int causal) {
    constexpr int NT = WM * WN * kWave;
    constexpr int TM = BM / WM, TN = BN / WN;
    constexpr int FM = TM / 32, FN = TN / 32;
    constexpr int LDS_K = BK + 8;
    constexpr int PASS = NT / BK;
    constexpr int A_PER_T = BM / PASS, B_PER_T = BN / PASS;
    static_assert(NT % BK == 0 && BM % PASS == 0 && BN % PASS == 0, "tile split");

    __shared__ __attribute__((aligned(16))) uint16_t As[BM * LDS_K];
    __shared__ __attribute__((aligned(16))) uint16_t Bs[BN * LDS_K];

    const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
    const int wm = wave / WN, wn = wave % WN;
    const int bh = blockIdx.z, b = bh / H, h = bh % H, g = h / (H / Hkv);
    const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
    const int off = Lk - Lq;
    const uint16_t *Qh = Q + static_cast<int64_t>(bh) * Lq * D;
    const uint16_t *Kh = Kc + (static_cast<int64_t>(b) * Hkv + g) * Lk * D;
    const int32_t *I = idx + static_cast<int64_t>(bh) * k;
    uint16_t *Sh = S + static_cast<int64_t>(bh) * Lq * Lk;

    if (causal && n0 > m0 + BM - 1 + off) {          // wholly masked tile
        for (int v = tid; v < BM * BN; v += NT) {
            const int m = m0 + v / BN, n = n0 + v % BN;
            if (m < Lq && n < Lk) Sh[static_cast<int64_t>(m) * Lk + n] = kBf16NegInf;
        }
        return;
    }

    const int a_t = tid % BK, row0 = tid / BK;
    uint16_t a_reg[A_PER_T], b_reg[B_PER_T];
    auto fetch = [&](int t0) {
        const int t = t0 + a_t;
        const int j = t < k ? I[t] : -1;
#pragma unroll
        for (int i = 0; i < A_PER_T; ++i) {
            const int m = m0 + row0 + i * PASS;
            a_reg[i] = (j >= 0 && m < Lq) ? Qh[static_cast<int64_t>(m) * D + j] : uint16_t(0);
        }
#pragma unroll
        for (int i = 0; i < B_PER_T; ++i) {
            const int n = n0 + row0 + i * PASS;
            b_reg[i] = (j >= 0 && n < Lk) ? Kh[static_cast<int64_t>(n) * D + j] : uint16_t(0);
        }
    };
    auto stash = [&]() {
#pragma unroll
        for (int i = 0; i < A_PER_T; ++i) As[(row0 + i * PASS) * LDS_K + a_t] = a_reg[i];
#pragma unroll
        for (int i = 0; i < B_PER_T; ++i) Bs[(row0 + i * PASS) * LDS_K + a_t] = b_reg[i];
    };

    f32x16_t acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    const int lr = lane % 32, lk = (lane / 32) * 8;
    fetch(0);
    for (int t0 = 0; t0 < k; t0 += BK) {
        stash();
        __syncthreads();
        if (t0 + BK < k) fetch(t0 + BK);
#pragma unroll
        for (int ks = 0; ks < BK; ks += 16) {
            bf16x8_t a[FM], bb[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i)
                a[i] = *reinterpret_cast<const bf16x8_t *>(&As[(wm * TM + i * 32 + lr) * LDS_K + ks + lk]);
#pragma unroll
            for (int j = 0; j < FN; ++j)
                bb[j] = *reinterpret_cast<const bf16x8_t *>(&Bs[(wn * TN + j * 32 + lr) * LDS_K + ks + lk]);
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], bb[j], acc[i][j], 0, 0, 0);
        }
        __syncthreads();
    }

#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const int n = n0 + wn * TN + j * 32 + lr;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int m = m0 + wm * TM + i * 32 + 8 * (v / 4) + 4 * (lane / 32) + (v % 4);
                if (m < Lq && n < Lk) {
                    const bool masked = causal && n > m + off;
                    Sh[static_cast<int64_t>(m) * Lk + n] =
                        masked ? kBf16NegInf : f32_to_bf16(acc[i][j][v] * scale);
                }
            }
        }
}

template <int BM, int BN, int BK>
__global__ __launch_bounds__(256) void qk_f32_kernel(
    const float *__restrict__ Q, const float *__restrict__ Kc, const int32_t *__restrict__ idx,
    float *__restrict__ S, int H, int Hkv, int Lq, int Lk, int D, int k, float scale, int causal) {
    constexpr int TX = 16, TY = 16;
    constexpr int RM = BM / TY, RN = BN / TX;
    __shared__ float As[BK][BM + 1];
    __shared__ float Bs[BK][BN + 1];
    const int tid = threadIdx.x, tx = tid % TX, ty = tid / TX;
    const int bh = blockIdx.z, b = bh / H, h = bh % H, g = h / (H / Hkv);
    const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
    const int off = Lk - Lq;
    const float *Qh = Q + static_cast<int64_t>(bh) * Lq * D;
    const float *Kh = Kc + (static_cast<int64_t>(b) * Hkv + g) * Lk * D;
    const int32_t *I = idx + static_cast<int64_t>(bh) * k;
    float *Sh = S + static_cast<int64_t>(bh) * Lq * Lk;

    float acc[RM][RN];
#pragma unroll
    for (int i = 0; i < RM; ++i)
#pragma unroll
        for (int j = 0; j < RN; ++j) acc[i][j] = 0.f;

    const bool skip = causal && n0 > m0 + BM - 1 + off;
    for (int t0 = 0; t0 < k && !skip; t0 += BK) {
        for (int v = tid; v < BM * BK; v += 256) {
            const int c = v % BK, r = v / BK;
            const int t = t0 + c, m = m0 + r;
            As[c][r] = (t < k && m < Lq) ? Qh[static_cast<int64_t>(m) * D + I[t]] : 0.f;
        }
        for (int v = tid; v < BN * BK; v += 256) {
            const int c = v % BK, r = v / BK;
            const int t = t0 + c, n = n0 + r;
            Bs[c][r] = (t < k && n < Lk) ? Kh[static_cast<int64_t>(n) * D + I[t]] : 0.f;
        }
        __syncthreads();
#pragma unroll
        for (int c = 0; c < BK; ++c) {
            float a[RM], bb[RN];
#pragma unroll
            for (int i = 0; i < RM; ++i) a[i] = As[c][ty + i * TY];
#pragma unroll
            for (int j = 0; j < RN; ++j) bb[j] = Bs[c][tx + j * TX];
#pragma unroll
            for (int i = 0; i < RM; ++i)
#pragma unroll
                for (int j = 0; j < RN; ++j) acc[i][j] = fmaf(a[i], bb[j], acc[i][j]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < RM; ++i)
#pragma unroll
        for (int j = 0; j < RN; ++j) {
            const int m = m0 + ty + i * TY, n = n0 + tx + j * TX;
            if (m < Lq && n < Lk)
                Sh[static_cast<int64_t>(m) * Lk + n] =
                    (causal && n > m + off) ? -__builtin_inff() : acc[i][j] * scale;
        }
}

}  // namespace

hipError_t launch_qk_bf16(const uint16_t *Q, const uint16_t *Kc, const int32_t *idx,
                          int64_t batch, int64_t H, int64_t Hkv, int64_t Lq, int64_t Lk,
                          int64_t D, int64_t k, float scale, bool causal, uint16_t *S,
                          hipStream_t stream) {
    constexpr int BM = 128, BN = 128, BK = 32, WM = 2, WN = 2;
    dim3 grid(static_cast<unsigned>((Lk + BN - 1) / BN), static_cast<unsigned>((Lq + BM - 1) / BM),
              static_cast<unsigned>(batch * H));
    hipLaunchKernelGGL((qk_bf16_kernel<BM, BN, BK, WM, WN>), grid, dim3(WM * WN * kWave), 0, stream,
                       Q, Kc, idx, S, static_cast<int>(H), static_cast<int>(Hkv),
                       static_cast<int>(Lq), static_cast<int>(Lk), static_cast<int>(D),
                       static_cast<int>(k), scale, causal ? 1 : 0);
    return hipGetLastError();
}

hipError_t launch_qk_f32(const float *Q, const float *Kc, const int32_t *idx, int64_t batch,
                         int64_t H, int64_t Hkv, int64_t Lq, int64_t Lk, int64_t D, int64_t k,
                         float scale, bool causal, float *S, hipStream_t stream) {
    constexpr int BM = 64, BN = 64, BK = 16;
    dim3 grid(static_cast<unsigned>((Lk + BN - 1) / BN), static_cast<unsigned>((Lq + BM - 1) / BM),
              static_cast<unsigned>(batch * H));
    hipLaunchKernelGGL((qk_f32_kernel<BM, BN, BK>), grid, dim3(256), 0, stream, Q, Kc, idx, S,
                       static_cast<int>(H), static_cast<int>(Hkv), static_cast<int>(Lq),
                       static_cast<int>(Lk), static_cast<int>(D), static_cast<int>(k), scale,
                       causal ? 1 : 0);
    return hipGetLastError();
}

}  // namespace rmm
