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
// Two launches.  rms_rowscale_kernel: one wave per row reads the row once
// (16-byte loads, fp32 sums of the exact squares in a fixed order, then an
// xor butterfly) and writes r_m.  Then the scoring pass's transposing tile
// kernel with its normalising variant: it reads X again (for the layer
// shapes the rows were just read and sit in the 256 MB Infinity Cache),
// normalises each value in registers, and writes the K-major copy as whole
// 128-byte row segments together with the float64 column energies.  The
// row statistic needs a whole row before any output of that row exists,
// which is why the rows are read twice; the row-major normalised rows are
// never written.
#include "device_common.h"
#include "kernels.h"

namespace rmm {

namespace {

constexpr int kRowThreads = 256;   // four rows per workgroup, one per wave

__global__ __launch_bounds__(kRowThreads) void rms_rowscale_kernel(
    const uint16_t *__restrict__ X, int64_t rows, int K, int64_t ldx, float eps,
    float *__restrict__ rscale) {
    const int lane = threadIdx.x & 63;
    const int64_t row = static_cast<int64_t>(blockIdx.x) * (kRowThreads / 64) + (threadIdx.x >> 6);
    if (row >= rows) return;                   // whole waves leave together
    const uint16_t *x = X + row * ldx;
    const int kc = K / 8;
    float s = 0.f;
    // eight 16-byte loads in flight per lane, added in chunk order
    for (int c0 = lane; c0 < kc; c0 += 8 * 64) {
        uint4 q[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int ch = c0 + 64 * i;
            q[i] = ch < kc ? *reinterpret_cast<const uint4 *>(x + 8 * ch) : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const uint32_t wd[4] = {q[i].x, q[i].y, q[i].z, q[i].w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float a = __uint_as_float(wd[e] << 16), b = __uint_as_float(wd[e] & 0xffff0000u);
                s = fmaf(a, a, s);
                s = fmaf(b, b, s);
            }
        }
    }
#pragma unroll
    for (int sh = 1; sh < 64; sh <<= 1) s += __shfl_xor(s, sh);
    if (lane == 0) rscale[row] = rsqrtf(s / static_cast<float>(K) + eps);
}

}  // namespace

size_t rmsnorm_workspace_bytes(int64_t B, int64_t M, int64_t K) {
    const size_t rs = (static_cast<size_t>(B * M) * sizeof(float) + 255) & ~static_cast<size_t>(255);
    return rs + score_workspace_bytes(B, M, K);
}

hipError_t launch_rmsnorm_kmajor(const uint16_t *X, const uint16_t *gamma, float eps, int64_t B,
                                 int64_t M, int64_t K, int64_t ldx, uint16_t *Xt, int64_t ldxt,
                                 double *energy, void *workspace, hipStream_t stream) {
    float *rscale = static_cast<float *>(workspace);
    double *partials = reinterpret_cast<double *>(
        static_cast<char *>(workspace) +
        ((static_cast<size_t>(B * M) * sizeof(float) + 255) & ~static_cast<size_t>(255)));
    // units are packed (unit stride M * ldx), so the B*M rows are one list
    const int64_t rows = B * M;
    const int64_t per = kRowThreads / 64;
    hipLaunchKernelGGL(rms_rowscale_kernel, dim3(static_cast<unsigned>((rows + per - 1) / per)),
                       dim3(kRowThreads), 0, stream, X, rows, static_cast<int>(K), ldx, eps, rscale);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_score_norm_kmajor(X, B, M, K, ldx, rscale, gamma, energy, partials, Xt, ldxt, stream);
}

}  // namespace rmm
