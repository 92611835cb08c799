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
// The row statistic needs a whole row before any output of that row exists,
// while the K-major copy is written in pieces of consecutive rows.
//
// K <= 4096: one pass.  rms_block_kmajor_kernel holds a block of 32 whole
// rows in registers (512 threads, up to 512 bytes each): it reads the block
// once, forms each row's scale from a fixed-order sum, normalises in
// registers, writes the block's K-major columns as 64-byte pieces (32
// tokens) and one float64 partial energy per (block, column), which a
// second kernel adds over the blocks in a fixed order (16 runs of
// consecutive blocks, each in order, then the runs in order).  The two
// blocks that share each 128-byte line of an Xt row run on the same XCD, so
// its L2 joins the halves.
//
// Wider rows: two launches.  rms_rowscale_kernel: one wave per row reads
// the row once (16-byte loads, fp32 sums of the exact squares in a fixed
// order, then an xor butterfly) and writes r_m.  Then the scoring pass's
// transposing tile kernel with its normalising variant reads X again (for
// the layer shapes the rows were just read and sit in the 256 MB Infinity
// Cache), normalises each value in registers, and writes the K-major copy as
// whole 128-byte row segments together with the float64 column energies.
// Either way the row-major normalised rows are never written.
#include <algorithm>

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


// ---------------------------------------------------------------- one pass
constexpr int kBlkRows = 32;                  // rows per workgroup
constexpr int kBlkWaves = 8, kBlkThreads = 64 * kBlkWaves;
constexpr int kBlkCols = 128;                 // columns of one wave tile
constexpr int64_t kBlkMaxK = 4 * kBlkWaves * kBlkCols;

// Wave tiles of 32 rows x 128 columns, tile t of the block taken by wave
// t % 8.  Lane 16*mc + jc holds rows 8*mc .. 8*mc+7 and columns 8*jc ..
// 8*jc+7 of each of its TPW tiles (one 16-byte load per row).  Row sums:
// the lane's columns in tile order, the 16 lanes of a row group (xor
// butterfly), then the eight waves in order.  Per tile and column: the
// lane's 8 exact float64 squares in row order, then the four row groups
// (xor butterfly).  out[(unit * nblk + block) * K + j] receives the block's
// sum for column j (out = energy when there is one block).
template <int TPW>
__global__ __launch_bounds__(kBlkThreads) void rms_block_kmajor_kernel(
    const uint16_t *__restrict__ X, int64_t M, int K, int64_t ldx, float eps,
    const uint16_t *__restrict__ gamma, uint16_t *__restrict__ Xt, int64_t ldxt,
    double *__restrict__ out) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int jc = lane & 15, mc = lane >> 4;
    const int64_t nblk = gridDim.x, unit = blockIdx.y;
    // workgroups w and w + 8 run on the same XCD: give them the two blocks
    // whose 64-byte pieces fill the same 128-byte lines of the Xt rows
    int64_t blk = blockIdx.x;
    if (nblk % 16 == 0) {
        const int64_t x = blk % 8, i = blk / 8;
        blk = 2 * (8 * (i / 2) + x) + (i % 2);
    }
    const int64_t m0 = blk * kBlkRows;
    const int rows = static_cast<int>(min<int64_t>(kBlkRows, M - m0));
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t *>(X + (unit * M + m0) * ldx), 0, static_cast<uint32_t>(rows * ldx * 2),
        0x00020000);
    constexpr uint32_t kOut = 0x80000000u;

    uint4 v[TPW][8];
#pragma unroll
    for (int t = 0; t < TPW; ++t) {
        const int j = (wave + kBlkWaves * t) * kBlkCols + 8 * jc;   // K % 8 == 0: whole groups
#pragma unroll
        for (int r = 0; r < 8; ++r) {
            const uint32_t off = j < K ? static_cast<uint32_t>(((8 * mc + r) * ldx + j) * 2) : kOut;
            const auto q = __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0);
            v[t][r] = make_uint4(q[0], q[1], q[2], q[3]);
        }
    }
    // row sums of the exact squares (fp32); absent rows and columns are zeros
    float s[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
        s[r] = 0.f;
#pragma unroll
        for (int t = 0; t < TPW; ++t) {
            const uint32_t w[4] = {v[t][r].x, v[t][r].y, v[t][r].z, v[t][r].w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float a = __uint_as_float(w[e] << 16), b = __uint_as_float(w[e] & 0xffff0000u);
                s[r] = fmaf(a, a, s[r]);
                s[r] = fmaf(b, b, s[r]);
            }
        }
#pragma unroll
        for (int sh = 1; sh < 16; sh <<= 1) s[r] += __shfl_xor(s[r], sh);
    }
    // the packed values stay the only copy of the block: without this the
    // compiler keeps their unpacked fp32 forms alive until the normalisation
#pragma unroll
    for (int t = 0; t < TPW; ++t)
#pragma unroll
        for (int r = 0; r < 8; ++r)
            asm volatile("" : "+v"(v[t][r].x), "+v"(v[t][r].y), "+v"(v[t][r].z), "+v"(v[t][r].w));
    __shared__ float red[kBlkWaves][kBlkRows];
    if (jc == 0) {
#pragma unroll
        for (int r = 0; r < 8; ++r) red[wave][8 * mc + r] = s[r];
    }
    __syncthreads();
    float sc[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
        float tot = red[0][8 * mc + r];
#pragma unroll
        for (int w = 1; w < kBlkWaves; ++w) tot += red[w][8 * mc + r];
        // absent rows (past M) are zeros; with eps = 0 their scale would be
        // infinite and 0 * inf a NaN, so they take scale 0
        sc[r] = 8 * mc + r < rows ? rsqrtf(tot / static_cast<float>(K) + eps) : 0.f;
    }

    uint16_t *xt = Xt + unit * static_cast<int64_t>(K) * ldxt + m0 + 8 * mc;
    double *o = out + (unit * nblk + blk) * static_cast<int64_t>(K);
#pragma unroll
    for (int t = 0; t < TPW; ++t) {
        const int j = (wave + kBlkWaves * t) * kBlkCols + 8 * jc;
        if ((wave + kBlkWaves * t) * kBlkCols >= K) break;          // uniform per wave
        const bool live = j < K;
        float gm[8];
        {
            const uint4 g = live ? *reinterpret_cast<const uint4 *>(gamma + j) : make_uint4(0, 0, 0, 0);
            const uint32_t gw[4] = {g.x, g.y, g.z, g.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                gm[2 * e] = __uint_as_float(gw[e] << 16);
                gm[2 * e + 1] = __uint_as_float(gw[e] & 0xffff0000u);
            }
        }
        double acc[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] = 0.0;
#pragma unroll
        for (int r = 0; r < 8; ++r) {
            uint32_t w[4] = {v[t][r].x, v[t][r].y, v[t][r].z, v[t][r].w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float xa = __uint_as_float(w[e] << 16), xb = __uint_as_float(w[e] & 0xffff0000u);
                w[e] = pack_bf16x2(bf16_to_f32(f32_to_bf16(xa * sc[r])) * gm[2 * e],
                                   bf16_to_f32(f32_to_bf16(xb * sc[r])) * gm[2 * e + 1]);
                // rows past M: zeros times scale 0, adding nothing
                const double ya = static_cast<double>(__uint_as_float(w[e] << 16));
                const double yb = static_cast<double>(__uint_as_float(w[e] & 0xffff0000u));
                acc[2 * e] = fma(ya, ya, acc[2 * e]);
                acc[2 * e + 1] = fma(yb, yb, acc[2 * e + 1]);
            }
            v[t][r] = make_uint4(w[0], w[1], w[2], w[3]);
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            acc[e] += __shfl_xor(acc[e], 16);
            acc[e] += __shfl_xor(acc[e], 32);
        }
        if (mc == 0 && live) {
#pragma unroll
            for (int e = 0; e < 8; ++e) o[j + e] = acc[e];
        }
        // column e of the lane's 8 x 8 block: 16 bytes (8 tokens) of Xt row j + e
        if (live) {
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const uint32_t sel = (e & 1) ? 0x07060302u : 0x05040100u;
                uint32_t ow[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const uint32_t a = reinterpret_cast<const uint32_t *>(&v[t][2 * q])[e >> 1];
                    const uint32_t b = reinterpret_cast<const uint32_t *>(&v[t][2 * q + 1])[e >> 1];
                    ow[q] = __builtin_amdgcn_perm(b, a, sel);
                }
                uint16_t *dst = xt + static_cast<int64_t>(j + e) * ldxt;
                if (8 * mc + 8 <= rows) {
                    *reinterpret_cast<uint4 *>(dst) = make_uint4(ow[0], ow[1], ow[2], ow[3]);
                } else {
#pragma unroll
                    for (int r = 0; r < 8; ++r)
                        if (8 * mc + r < rows) dst[r] = static_cast<uint16_t>(ow[r >> 1] >> (16 * (r & 1)));
                }
            }
        }
    }
}

}  // namespace

// a block's rows are addressed with 32-bit byte offsets
bool rmsnorm_single_pass(int64_t K, int64_t ldx) {
    return K <= kBlkMaxK && kBlkRows * ldx * 2 < (int64_t(1) << 31);
}

// enough for either path (the path also depends on ldx)
size_t rmsnorm_workspace_bytes(int64_t B, int64_t M, int64_t K) {
    const int64_t nblk = (M + kBlkRows - 1) / kBlkRows;
    const size_t one = K <= kBlkMaxK && nblk > 1 ? static_cast<size_t>(B * nblk * K) * sizeof(double) : 0;
    const size_t rs = (static_cast<size_t>(B * M) * sizeof(float) + 255) & ~static_cast<size_t>(255);
    return std::max(one, rs + score_workspace_bytes(B, M, K));
}

hipError_t launch_rmsnorm_kmajor(const uint16_t *X, const uint16_t *gamma, float eps, int64_t B,
                                 int64_t M, int64_t K, int64_t ldx, uint16_t *Xt, int64_t ldxt,
                                 double *energy, void *workspace, hipStream_t stream) {
    if (rmsnorm_single_pass(K, ldx)) {
        const int64_t nblk = (M + kBlkRows - 1) / kBlkRows;
        double *out = nblk > 1 ? static_cast<double *>(workspace) : energy;
        const int tiles = static_cast<int>((K + kBlkCols - 1) / kBlkCols);
        const int tpw = (tiles + kBlkWaves - 1) / kBlkWaves;
        const dim3 grid(static_cast<unsigned>(nblk), static_cast<unsigned>(B));
        const int Ki = static_cast<int>(K);
        auto launch = [&](auto kernel) {
            hipLaunchKernelGGL(kernel, grid, dim3(kBlkThreads), 0, stream, X, M, Ki, ldx, eps, gamma,
                               Xt, ldxt, out);
        };
        switch (tpw) {          // column tiles per wave
        case 1: launch(rms_block_kmajor_kernel<1>); break;
        case 2: launch(rms_block_kmajor_kernel<2>); break;
        case 3: launch(rms_block_kmajor_kernel<3>); break;
        default: launch(rms_block_kmajor_kernel<4>); break;
        }
        hipError_t e = hipGetLastError();
        if (e != hipSuccess || nblk == 1) return e;
        return launch_score_finalize_grouped(out, B, nblk, K, energy, stream);
    }
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
