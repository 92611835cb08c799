// Gathered reduced product Y = X[:, I] W[I, :]   (Sec. 3.2 definition of
// RMM; Sec. 3.3 projections).
//
// bf16 path: MFMA GEMM (v_mfma_f32_32x32x16_bf16, fp32 accumulate) whose
// K-loop walks the retained index list.  Each k-tile of BK retained indices
// is gathered straight from the uncompacted operands into LDS:
//   * X[m, I(t)]: lanes run along t within one row, so a wave's 2-byte loads
//     fall in the few cache lines that hold that row's retained columns;
//   * W[I(t), n0:n0+BN]: whole 16-byte row vectors, written to LDS transposed
//     (n-major) so both MFMA operands read 8 consecutive t per lane.
// The next k-tile is fetched into registers while the current one is
// multiplied.  Index tails (k not a multiple of BK) and M/N tails are zero-
// filled; no compacted copy of either operand is ever written to memory.
//
// fp32 path: the same gather into LDS with a VALU FMA tile (fp32 accumulate).
#include "device_common.h"
#include "kernels.h"

namespace rmm {

namespace {

// ------------------------------------------------------------------ bf16
template <int BM, int BN, int BK, int WM, int WN, bool VECW>
__global__ __launch_bounds__(WM *WN *kWave) void gemm_gather_bf16_kernel(
    const uint16_t *__restrict__ X, const uint16_t *__restrict__ W,
    const int32_t *__restrict__ idx, uint16_t *__restrict__ Y, int M, int N, int k,
    int64_t ldx, int64_t ldw, int64_t ldy) {
    constexpr int NT = WM * WN * kWave;
    constexpr int TM = BM / WM, TN = BN / WN;        // per-wave tile
    constexpr int FM = TM / 32, FN = TN / 32;        // 32x32 fragments per wave
    constexpr int LDS_K = BK + 8;                    // padded row (elements)
    constexpr int A_PER_T = BM * BK / NT;            // gathered X elements per thread
    constexpr int ROWS_PER_PASS = NT / BK;
    constexpr int VPR = BN / 8;                      // 16-byte vectors per W row
    constexpr int W_PER_T = BK * VPR / NT;
    static_assert(BM * BK % NT == 0 && NT % BK == 0, "A tile split");
    static_assert(BK * VPR % NT == 0, "W tile split");
    static_assert(TM % 32 == 0 && TN % 32 == 0 && BK % 16 == 0, "fragments");

    __shared__ __attribute__((aligned(16))) uint16_t As[BM * LDS_K];
    __shared__ __attribute__((aligned(16))) uint16_t Bs[BN * LDS_K];

    const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
    const int wm = wave / WN, wn = wave % WN;
    const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
    const int64_t unit = blockIdx.z;
    X += unit * static_cast<int64_t>(M) * ldx;
    Y += unit * static_cast<int64_t>(M) * ldy;
    idx += unit * k;

    const int a_t = tid % BK;                 // retained position within the tile
    const int a_row0 = tid / BK;

    uint16_t a_reg[A_PER_T];
    uint4 w_reg[W_PER_T];

    auto fetch = [&](int t0) {
        const int ta = t0 + a_t;
        const int ja = ta < k ? idx[ta] : -1;
#pragma unroll
        for (int i = 0; i < A_PER_T; ++i) {
            const int m = m0 + a_row0 + i * ROWS_PER_PASS;
            a_reg[i] = (ja >= 0 && m < M) ? X[static_cast<int64_t>(m) * ldx + ja] : uint16_t(0);
        }
#pragma unroll
        for (int i = 0; i < W_PER_T; ++i) {
            const int v = tid + i * NT;
            const int c = v / VPR, seg = v % VPR;
            const int tc = t0 + c;
            const int jw = tc < k ? idx[tc] : -1;
            const int n = n0 + seg * 8;
            uint4 w = make_uint4(0, 0, 0, 0);
            if (jw >= 0) {
                const uint16_t *p = W + static_cast<int64_t>(jw) * ldw + n;
                if (VECW && n + 8 <= N) {
                    w = *reinterpret_cast<const uint4 *>(p);
                } else {
                    uint16_t tmp[8];
#pragma unroll
                    for (int e = 0; e < 8; ++e) tmp[e] = (n + e < N) ? p[e] : uint16_t(0);
                    w = *reinterpret_cast<const uint4 *>(tmp);
                }
            }
            w_reg[i] = w;
        }
    };
    auto stash = [&]() {
#pragma unroll
        for (int i = 0; i < A_PER_T; ++i) As[(a_row0 + i * ROWS_PER_PASS) * LDS_K + a_t] = a_reg[i];
#pragma unroll
        for (int i = 0; i < W_PER_T; ++i) {
            const int v = tid + i * NT;
            const int c = v / VPR, seg = v % VPR;
            const uint16_t *e8 = reinterpret_cast<const uint16_t *>(&w_reg[i]);
#pragma unroll
            for (int e = 0; e < 8; ++e) Bs[(seg * 8 + e) * LDS_K + c] = e8[e];
        }
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
            bf16x8_t a[FM], b[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i)
                a[i] = *reinterpret_cast<const bf16x8_t *>(&As[(wm * TM + i * 32 + lr) * LDS_K + ks + lk]);
#pragma unroll
            for (int j = 0; j < FN; ++j)
                b[j] = *reinterpret_cast<const bf16x8_t *>(&Bs[(wn * TN + j * 32 + lr) * LDS_K + ks + lk]);
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
        }
        __syncthreads();
    }

    // C fragment: lane holds column lr, rows 8*(v/4) + 4*(lane/32) + v%4
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const int n = n0 + wn * TN + j * 32 + lr;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int m = m0 + wm * TM + i * 32 + 8 * (v / 4) + 4 * (lane / 32) + (v % 4);
                if (m < M && n < N) Y[static_cast<int64_t>(m) * ldy + n] = f32_to_bf16(acc[i][j][v]);
            }
        }
}

// ------------------------------------------------------------------ fp32
template <int BM, int BN, int BK>
__global__ __launch_bounds__(256) void gemm_gather_f32_kernel(
    const float *__restrict__ X, const float *__restrict__ W, const int32_t *__restrict__ idx,
    float *__restrict__ Y, int M, int N, int k, int64_t ldx, int64_t ldw, int64_t ldy) {
    constexpr int TX = 16, TY = 16;                  // 256 threads
    constexpr int RM = BM / TY, RN = BN / TX;        // outputs per thread
    __shared__ float As[BK][BM + 1];
    __shared__ float Bs[BK][BN + 1];
    const int tid = threadIdx.x, tx = tid % TX, ty = tid / TX;
    const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
    const int64_t unit = blockIdx.z;
    X += unit * static_cast<int64_t>(M) * ldx;
    Y += unit * static_cast<int64_t>(M) * ldy;
    idx += unit * k;

    float acc[RM][RN];
#pragma unroll
    for (int i = 0; i < RM; ++i)
#pragma unroll
        for (int j = 0; j < RN; ++j) acc[i][j] = 0.f;

    for (int t0 = 0; t0 < k; t0 += BK) {
        // X tile: lanes along the retained position within one row
        for (int v = tid; v < BM * BK; v += 256) {
            const int c = v % BK, r = v / BK;
            const int t = t0 + c, m = m0 + r;
            As[c][r] = (t < k && m < M) ? X[static_cast<int64_t>(m) * ldx + idx[t]] : 0.f;
        }
        for (int v = tid; v < BK * BN; v += 256) {
            const int c = v / BN, n = v % BN;
            const int t = t0 + c;
            Bs[c][n] = (t < k && n0 + n < N) ? W[static_cast<int64_t>(idx[t]) * ldw + n0 + n] : 0.f;
        }
        __syncthreads();
#pragma unroll
        for (int c = 0; c < BK; ++c) {
            float a[RM], b[RN];
#pragma unroll
            for (int i = 0; i < RM; ++i) a[i] = As[c][ty + i * TY];
#pragma unroll
            for (int j = 0; j < RN; ++j) b[j] = Bs[c][tx + j * TX];
#pragma unroll
            for (int i = 0; i < RM; ++i)
#pragma unroll
                for (int j = 0; j < RN; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < RM; ++i)
#pragma unroll
        for (int j = 0; j < RN; ++j) {
            const int m = m0 + ty + i * TY, n = n0 + tx + j * TX;
            if (m < M && n < N) Y[static_cast<int64_t>(m) * ldy + n] = acc[i][j];
        }
}

}  // namespace

hipError_t launch_gemm_bf16(const uint16_t *X, const uint16_t *W, const int32_t *idx,
                            int64_t B, int64_t M, int64_t N, int64_t K, int64_t k,
                            int64_t ldx, int64_t ldw, uint16_t *Y, int64_t ldy,
                            hipStream_t stream) {
    (void)K;
    constexpr int BM = 128, BN = 128, BK = 32, WM = 2, WN = 2;
    dim3 grid(static_cast<unsigned>((N + BN - 1) / BN), static_cast<unsigned>((M + BM - 1) / BM),
              static_cast<unsigned>(B));
    const bool vec = (reinterpret_cast<uintptr_t>(W) % 16 == 0) && (ldw % 8 == 0);
    if (vec)
        hipLaunchKernelGGL((gemm_gather_bf16_kernel<BM, BN, BK, WM, WN, true>), grid,
                           dim3(WM * WN * kWave), 0, stream, X, W, idx, Y, static_cast<int>(M),
                           static_cast<int>(N), static_cast<int>(k), ldx, ldw, ldy);
    else
        hipLaunchKernelGGL((gemm_gather_bf16_kernel<BM, BN, BK, WM, WN, false>), grid,
                           dim3(WM * WN * kWave), 0, stream, X, W, idx, Y, static_cast<int>(M),
                           static_cast<int>(N), static_cast<int>(k), ldx, ldw, ldy);
    return hipGetLastError();
}

hipError_t launch_gemm_f32(const float *X, const float *W, const int32_t *idx, int64_t B,
                           int64_t M, int64_t N, int64_t K, int64_t k, int64_t ldx, int64_t ldw,
                           float *Y, int64_t ldy, hipStream_t stream) {
    (void)K;
    constexpr int BM = 64, BN = 64, BK = 16;
    dim3 grid(static_cast<unsigned>((N + BN - 1) / BN), static_cast<unsigned>((M + BM - 1) / BM),
              static_cast<unsigned>(B));
    hipLaunchKernelGGL((gemm_gather_f32_kernel<BM, BN, BK>), grid, dim3(256), 0, stream, X, W, idx, Y,
                       static_cast<int>(M), static_cast<int>(N), static_cast<int>(k), ldx, ldw, ldy);
    return hipGetLastError();
}

}  // namespace rmm
