// RMSNorm producing a reduced projection's input in the K-major form the
// gathered GEMM reads, with that input's column energies (Sec. 3.2 scores
// from the projection's own input; the Limitations section names the memory
// movement of a separate scoring pass as a cost to remove).
//
//   r_m            = 1 / sqrt(mean_j X[m][j]^2 + eps)          (fp32)
//   y[m][j]        = bf16(gamma_j * bf16(X[m][j] * r_m))       (as the model's
//                    norm stores its bf16 output, then scales by its weight)
//   Xt[j][m]       = y[m][j]
//   energy[j]      = sum over m of y[m][j]^2                   (float64, exact
//                    squares, fixed order)
//
// HBM-bound; X is read once.  A workgroup stages R whole rows (R*K*2 bytes,
// at most 128 KiB) in LDS, takes the rows' statistics, then writes the
// block's K x R transpose: each thread owns 8 channels and emits, per 8 rows,
// one 16-byte piece of each of its 8 Xt rows.  The global loads of the next
// block go out before the current block's stores, into registers.  Blocks
// are dealt so that the workgroups of one XCD hold consecutive row blocks at
// the same time: the 2R-byte pieces of one Xt line then meet in that XCD's
// L2 before the line is written back.  Column energies are summed per thread
// over its blocks in order, then per workgroup in order by the finalize
// kernel.  No atomics: results are bit-reproducible.
#include <type_traits>

#include "device_common.h"
#include "kernels.h"

namespace rmm {

namespace {

constexpr int kNormThreads = 512;
constexpr int kNormLdsElems = 65536;          // 128 KiB of staged bf16 rows
// R rows per block, G 8-channel groups per thread (8 * G * kNormThreads >= K)
template <int R, int G>
__global__ __launch_bounds__(kNormThreads, 1) void rmsnorm_kmajor_kernel(
    const uint16_t *__restrict__ X, int64_t M, int K, int64_t ldx, const uint16_t *__restrict__ gamma,
    float eps, uint16_t *__restrict__ Xt, int64_t ldxt, double *__restrict__ part, int64_t nblk) {
    static_assert(R % 8 == 0 && R >= 8 && G >= 1, "rows per block");
    __shared__ __attribute__((aligned(16))) uint16_t rows[kNormLdsElems];
    __shared__ float rinv[R];
    constexpr int kLoads = kNormLdsElems / 8 / kNormThreads;   // 16-byte chunks per thread

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int W = gridDim.x, w = blockIdx.x;
    const int64_t unit = blockIdx.y;
    const int kc = K / 8;                         // 16-byte chunks per row
    const int nchunks = R * kc;                   // chunks per block (<= 8192)
    X += unit * M * ldx;
    Xt += unit * static_cast<int64_t>(K) * ldxt;
    // XCD x (workgroups w % 8 == x) takes the W/8 consecutive blocks
    // it*W + x*W/8 .. of every round `it`
    const int64_t slot = (W % 8 == 0) ? (w % 8) * (W / 8) + w / 8 : w;

    double acc[G][8];
#pragma unroll
    for (int q = 0; q < G; ++q)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[q][e] = 0.0;
    uint4 g8[G];
#pragma unroll
    for (int q = 0; q < G; ++q) {
        const int g = tid + q * kNormThreads;
        g8[q] = g < kc ? *reinterpret_cast<const uint4 *>(gamma + 8 * g) : make_uint4(0, 0, 0, 0);
    }

    uint4 v[kLoads];
    // loads i0 .. i1-1 of a block's chunks into v
    auto load = [&](int64_t blk, auto I0, auto I1) {
        const int64_t m0 = blk * R;
#pragma unroll
        for (int i = decltype(I0)::value; i < decltype(I1)::value; ++i) {
            const int c = tid + i * kNormThreads;
            const int r = c / kc, ch = c - r * kc;
            const int64_t m = m0 + r;
            v[i] = (c < nchunks && m < M)
                ? *reinterpret_cast<const uint4 *>(X + m * ldx + 8 * ch) : make_uint4(0, 0, 0, 0);
        }
    };

    using L0 = std::integral_constant<int, 0>;
    // loads of the next block issued before this one's stores: half of them,
    // a quarter with two channel groups per thread (register budget)
    using LH = std::integral_constant<int, G == 1 ? kLoads / 2 : kLoads / 4>;
    using L1 = std::integral_constant<int, kLoads>;
    int64_t blk = slot;
    if (blk < nblk) load(blk, L0{}, LH{});
    for (; blk < nblk; blk += W) {
        const int64_t m0 = blk * R;
        load(blk, LH{}, L1{});
        // stage the block (row r at rows[r*K])
#pragma unroll
        for (int i = 0; i < kLoads; ++i) {
            const int c = tid + i * kNormThreads;
            if (c < nchunks) *reinterpret_cast<uint4 *>(&rows[8 * c]) = v[i];
        }
        __syncthreads();
        // row statistics: wave w takes rows w, w+8, ...; lanes add their
        // chunks in order, then an xor butterfly (every lane ends with the
        // same sum)
        for (int r = wave; r < R; r += kNormThreads / 64) {
            float s = 0.f;
            for (int ch = lane; ch < kc; ch += 64) {
                const uint4 q = *reinterpret_cast<const uint4 *>(&rows[r * K + 8 * ch]);
                const uint32_t wd[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float a = __uint_as_float(wd[e] << 16), b = __uint_as_float(wd[e] & 0xffff0000u);
                    s = fmaf(a, a, s);
                    s = fmaf(b, b, s);
                }
            }
#pragma unroll
            for (int sh = 1; sh < 64; sh <<= 1) s += __shfl_xor(s, sh);
            if (lane == 0) rinv[r] = rsqrtf(s / static_cast<float>(K) + eps);
        }
        __syncthreads();
        if (blk + W < nblk) load(blk + W, L0{}, LH{});
#pragma unroll
        for (int q = 0; q < G; ++q) {
            const int g = tid + q * kNormThreads;
            if (g >= kc) continue;
            const uint32_t gw[4] = {g8[q].x, g8[q].y, g8[q].z, g8[q].w};
#pragma unroll 1
            for (int r8 = 0; r8 < R; r8 += 8) {
                uint32_t yv[8][4];          // [row][packed channel pair]
#pragma unroll
                for (int rr = 0; rr < 8; ++rr) {
                    const int r = r8 + rr;
                    const uint4 xq = *reinterpret_cast<const uint4 *>(&rows[r * K + 8 * g]);
                    const uint32_t xw[4] = {xq.x, xq.y, xq.z, xq.w};
                    const float rv = m0 + r < M ? rinv[r] : 0.f;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float xa = __uint_as_float(xw[e] << 16), xb = __uint_as_float(xw[e] & 0xffff0000u);
                        const float ga = __uint_as_float(gw[e] << 16), gb = __uint_as_float(gw[e] & 0xffff0000u);
                        const float ya = bf16_to_f32(f32_to_bf16(bf16_to_f32(f32_to_bf16(xa * rv)) * ga));
                        const float yb = bf16_to_f32(f32_to_bf16(bf16_to_f32(f32_to_bf16(xb * rv)) * gb));
                        yv[rr][e] = pack_bf16x2(ya, yb);
                        const double da = static_cast<double>(ya), db = static_cast<double>(yb);
                        acc[q][2 * e] = fma(da, da, acc[q][2 * e]);
                        acc[q][2 * e + 1] = fma(db, db, acc[q][2 * e + 1]);
                    }
                }
                // channel e of the 8 x 8 block -> one 16-byte piece of Xt row 8g + e
                const int64_t mrow = m0 + r8;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const uint32_t sel = (e & 1) ? 0x07060302u : 0x05040100u;
                    uint32_t o[4];
#pragma unroll
                    for (int p = 0; p < 4; ++p) o[p] = __builtin_amdgcn_perm(yv[2 * p + 1][e >> 1], yv[2 * p][e >> 1], sel);
                    uint16_t *dst = Xt + static_cast<int64_t>(8 * g + e) * ldxt + mrow;
                    if (mrow + 8 <= M) {
                        *reinterpret_cast<uint4 *>(dst) = make_uint4(o[0], o[1], o[2], o[3]);
                    } else {
#pragma unroll
                        for (int rr = 0; rr < 8; ++rr)
                            if (mrow + rr < M) dst[rr] = static_cast<uint16_t>(o[rr >> 1] >> (16 * (rr & 1)));
                    }
                }
            }
        }
        __syncthreads();          // the block's rows are read before the next one lands
    }
    // this workgroup's share of the column energies, in the finalize layout
    double *pw = part + (unit * W + w) * static_cast<int64_t>(K);
#pragma unroll
    for (int q = 0; q < G; ++q) {
        const int g = tid + q * kNormThreads;
        if (g >= kc) continue;
#pragma unroll
        for (int e = 0; e < 8; ++e) pw[8 * g + e] = acc[q][e];
    }
}

}  // namespace

int rmsnorm_rows_per_block(int64_t K) {
    return K <= 2048 ? 32 : K <= 4096 ? 16 : 8;
}

int64_t rmsnorm_workgroups(int64_t B, int64_t M, int64_t K) {
    const int64_t nblk = (M + rmsnorm_rows_per_block(K) - 1) / rmsnorm_rows_per_block(K);
    // about one workgroup per CU over all units (one fits a CU: 128 KiB LDS)
    int64_t w = (256 + B - 1) / B;
    w = (w + 7) / 8 * 8;
    return w < nblk ? w : nblk;
}

size_t rmsnorm_workspace_bytes(int64_t B, int64_t M, int64_t K) {
    return static_cast<size_t>(B * rmsnorm_workgroups(B, M, K) * K) * sizeof(double);
}

hipError_t launch_rmsnorm_kmajor(const uint16_t *X, const uint16_t *gamma, float eps, int64_t B,
                                 int64_t M, int64_t K, int64_t ldx, uint16_t *Xt, int64_t ldxt,
                                 double *energy, double *partials, hipStream_t stream) {
    const int R = rmsnorm_rows_per_block(K);
    const int64_t nblk = (M + R - 1) / R;
    const int64_t W = rmsnorm_workgroups(B, M, K);
    dim3 grid(static_cast<unsigned>(W), static_cast<unsigned>(B));
    const int k32 = static_cast<int>(K);
    if (R == 32)
        hipLaunchKernelGGL((rmsnorm_kmajor_kernel<32, 1>), grid, dim3(kNormThreads), 0, stream, X, M, k32,
                           ldx, gamma, eps, Xt, ldxt, partials, nblk);
    else if (R == 16)
        hipLaunchKernelGGL((rmsnorm_kmajor_kernel<16, 1>), grid, dim3(kNormThreads), 0, stream, X, M, k32,
                           ldx, gamma, eps, Xt, ldxt, partials, nblk);
    else
        hipLaunchKernelGGL((rmsnorm_kmajor_kernel<8, 2>), grid, dim3(kNormThreads), 0, stream, X, M, k32,
                           ldx, gamma, eps, Xt, ldxt, partials, nblk);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_score_finalize(partials, B, W, K, energy, stream);
}

}  // namespace rmm
