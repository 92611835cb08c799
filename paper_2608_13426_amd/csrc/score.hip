// Column energies e_j = sum_m X[m][j]^2 of each selection unit
// (Sec. 3.2 score s_j = ||A[:, j]||_2, ranked through s_j^2).
//
// HBM-bound streaming reduction.  Each workgroup owns 128 columns of one row
// split of one unit; its lanes read whole 16-byte vectors along a row, so a
// wave touches full 128-byte lines.  bf16/fp32 values are squared exactly in
// float64 and accumulated in float64 in a fixed order: per thread over its
// rows, then the row groups of the workgroup in order, then the splits in
// order (second kernel).  No atomics, so results are bit-reproducible.
//
// Optionally the same pass writes a K-major copy Xt[b][j][m] = X[b][m][j]
// (bf16): each 64-row slab is staged in LDS and written out as whole
// 128-byte segments of Xt rows.  The gathered GEMM then reads a retained
// index as one contiguous Xt row.
#include "device_common.h"
#include "kernels.h"

namespace rmm {

namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ double to_f64(uint16_t v) { return static_cast<double>(bf16_to_f32(v)); }
__device__ __forceinline__ double to_f64(float v) { return static_cast<double>(v); }

// VEC = elements per 16-byte load, or 1 for the element-wise path used when
// rows are not 16-byte aligned.
// Slab layout for the transposed copy: 64 rows x 128 columns of bf16, row
// stride 136; column c of row r is stored at c ^ (8 * ((r >> 3) & 7)), so the
// column-wise reads of 8 rows 8 apart fall on distinct banks.
constexpr int kSlabRows = 64, kSlabStride = kScoreCols + 8;
__device__ __forceinline__ int slab_at(int r, int c) {
    return r * kSlabStride + (c ^ (8 * ((r >> 3) & 7)));
}

template <typename T, int VEC, bool XT>
__global__ __launch_bounds__(kThreads) void score_partial_kernel(
    const T *__restrict__ X, int64_t M, int64_t K, int64_t ldx, int64_t rows_per_split,
    double *__restrict__ out, int64_t out_unit_stride, int64_t out_split_stride,
    uint16_t *__restrict__ Xt, int64_t ldxt) {
    constexpr int TPR = kScoreCols / VEC;     // threads along a row
    constexpr int RPI = kThreads / TPR;       // rows per iteration
    static_assert(!XT || (VEC == 8 && 4 * RPI == kSlabRows), "transposed copy: bf16 vector path");
    __shared__ double red[RPI][kScoreCols];
    __shared__ __attribute__((aligned(16))) uint16_t slab[XT ? kSlabRows * kSlabStride : 1];

    const int tid = threadIdx.x;
    const int lane_col = (tid % TPR) * VEC;
    const int row_off = tid / TPR;
    const int64_t col0 = static_cast<int64_t>(blockIdx.x) * kScoreCols + lane_col;
    const int64_t split = blockIdx.y;
    const int64_t unit = blockIdx.z;
    const int64_t r_begin = split * rows_per_split;
    const int64_t r_end = min(M, r_begin + rows_per_split);
    const T *base = X + unit * M * ldx;

    double acc[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) acc[v] = 0.0;

    if constexpr (VEC > 1) {
        const bool full = col0 + VEC <= K;
        // whole 64-row slabs (a trip count uniform across the workgroup, as
        // the slab loop below synchronises), four rows in flight per thread
        const int64_t n_slabs = (r_end - r_begin) / (4 * RPI);
        int64_t r = r_begin + row_off;
        for (int64_t sl = 0; sl < n_slabs; ++sl, r += 4 * RPI) {
            uint4 q[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const T *p = base + (r + u * RPI) * ldx + col0;
                if (full) {
                    q[u] = *reinterpret_cast<const uint4 *>(p);
                } else {
                    T tmp[VEC];
#pragma unroll
                    for (int v = 0; v < VEC; ++v) tmp[v] = (col0 + v < K) ? p[v] : T(0);
                    q[u] = *reinterpret_cast<const uint4 *>(tmp);
                }
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const T *t = reinterpret_cast<const T *>(&q[u]);
#pragma unroll
                for (int v = 0; v < VEC; ++v) {
                    const double x = to_f64(t[v]);
                    acc[v] = fma(x, x, acc[v]);
                }
            }
            if constexpr (XT) {
                // stage the 64-row slab, then write 8 lanes per 128-byte Xt segment
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    *reinterpret_cast<uint4 *>(&slab[slab_at(row_off + u * RPI, lane_col)]) = q[u];
                __syncthreads();
                const int64_t slab_row0 = r - row_off;
                const int rq = (threadIdx.x & 7) * 8;          // 8 rows of the slab
#pragma unroll
                for (int pass = 0; pass < kScoreCols / 32; ++pass) {
                    const int c = pass * 32 + (threadIdx.x >> 3);
                    const int64_t col = static_cast<int64_t>(blockIdx.x) * kScoreCols + c;
                    uint32_t w[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        w[e] = static_cast<uint32_t>(slab[slab_at(rq + 2 * e, c)]) |
                               (static_cast<uint32_t>(slab[slab_at(rq + 2 * e + 1, c)]) << 16);
                    if (col < K)
                        *reinterpret_cast<uint4 *>(Xt + unit * K * ldxt + col * ldxt + slab_row0 + rq) =
                            make_uint4(w[0], w[1], w[2], w[3]);
                }
                __syncthreads();
            }
        }
        for (; r < r_end; r += RPI) {
            const T *p = base + r * ldx + col0;
#pragma unroll
            for (int v = 0; v < VEC; ++v) {
                const double x = (col0 + v < K) ? to_f64(p[v]) : 0.0;
                acc[v] = fma(x, x, acc[v]);
                if constexpr (XT) {
                    if (col0 + v < K) Xt[unit * K * ldxt + (col0 + v) * ldxt + r] = p[v];
                }
            }
        }
    } else {
        if (col0 < K) {
            for (int64_t r = r_begin + row_off; r < r_end; r += RPI) {
                const double x = to_f64(base[r * ldx + col0]);
                acc[0] = fma(x, x, acc[0]);
            }
        }
    }

#pragma unroll
    for (int v = 0; v < VEC; ++v) red[row_off][lane_col + v] = acc[v];
    __syncthreads();
    if (tid < kScoreCols) {
        double s = 0.0;
#pragma unroll
        for (int g = 0; g < RPI; ++g) s += red[g][tid];
        const int64_t col = static_cast<int64_t>(blockIdx.x) * kScoreCols + tid;
        if (col < K) out[unit * out_unit_stride + split * out_split_stride + col] = s;
    }
}

// bf16 rows with 16-byte aligned starts (ldx % 8 == 0): each wave reads a
// 64-row x 64-column tile as eight 16-byte row vectors per lane (lanes
// 8*mc + jc: rows 8*mc .. 8*mc+7, columns 8*jc .. 8*jc+7, so eight lanes
// cover one 128-byte row segment), squares them into float64 column sums,
// and, for the K-major copy, transposes its 8 x 8 block in registers and
// stores eight 16-byte Xt vectors (eight lanes cover one 128-byte segment
// of an Xt row).  The workgroup's four waves take consecutive tiles; their
// column sums are combined in a fixed order.  (16 column groups per wave,
// 32 x 128 tiles, measured faster for 4096 columns and slower for 14336.)
constexpr int kStrip = 64;      // columns per workgroup that set the split policy
constexpr int kTileJC = 8;      // 8-column groups per wave (8: 64 x 64 wave tiles)

// MODE 1 (RMSNorm): the values are first normalised as an RMSNorm stores
// them, y = bf16(gamma[j] * bf16(x * rscale[m])) with the row scale of each
// row (rscale: one float per row of every unit).  MODE 2 (softmax): the rows
// are attention scores and y = bf16(exp(x - rmax[m]) * rinv[m]) (rscale holds
// rmax, rinv2 the reciprocal row sums; rows of every unit in turn), zero
// where the causal mask drops (m, j) (causal != 0 and j > m + coff), whose
// scores are then never read; such zeros are stored in the K-major copy at
// least where m >= 256 * floor((j - coff) / 256) (the 256-row block of the
// column's diagonal: what a causal value product reads) and may be left
// unwritten before it (wave tiles wholly there store nothing).  The energies and the K-major copy are those
// of y.
template <bool XT, int JC, int MODE = 0>
__global__ __launch_bounds__(kThreads) void score_tile_kernel(
    const uint16_t *__restrict__ X, int64_t M, int64_t K, int64_t ldx, int64_t rows_per_split,
    double *__restrict__ out, int64_t out_unit_stride, int64_t out_split_stride,
    uint16_t *__restrict__ Xt, int64_t ldxt, const float *__restrict__ rscale = nullptr,
    const uint16_t *__restrict__ gamma = nullptr, const float *__restrict__ rinv2 = nullptr,
    int64_t coff = 0, int causal = 0) {
    constexpr bool NORM = MODE == 1, SOFTMAX = MODE == 2;
    constexpr int MC = 64 / JC, STRIP = 8 * JC, TROWS = 8 * MC;   // wave tile TROWS x STRIP
    __shared__ double red[kThreads / 64][STRIP];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int jc = lane % JC, mc = lane / JC;
    const int64_t j = static_cast<int64_t>(blockIdx.x) * STRIP + 8 * jc;
    const int64_t split = blockIdx.y, unit = blockIdx.z;
    const int64_t r_begin = split * rows_per_split;
    const int rows = static_cast<int>(min(M, r_begin + rows_per_split) - r_begin);
    const int nvalid = static_cast<int>(max<int64_t>(0, min<int64_t>(8, K - j)));
    // the split's rows as one buffer: rows past its end read zeros
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t *>(X + (unit * M + r_begin) * ldx), 0,
        static_cast<uint32_t>(rows * ldx * 2), 0x00020000);
    constexpr uint32_t kOut = 0x80000000u;
    const uint32_t col_off = nvalid > 0 ? static_cast<uint32_t>(j * 2) : kOut;
    uint16_t *xt = XT ? Xt + (unit * K + j) * ldxt + r_begin : nullptr;
    float gm[8];
    const float *rsu = MODE ? rscale + unit * M + r_begin : nullptr;
    const float *riu = SOFTMAX ? rinv2 + unit * M + r_begin : nullptr;
    if constexpr (NORM) {
#pragma unroll
        for (int e = 0; e < 8; ++e) gm[e] = e < nvalid ? bf16_to_f32(gamma[j + e]) : 0.f;
    }

    double acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.0;
    for (int m0 = wave * TROWS; m0 < rows; m0 += 4 * TROWS) {
        uint4 v[8];
        // softmax with the causal mask: a wave tile whose every key lies
        // past its last query's limit reads nothing
        const int64_t j_first = static_cast<int64_t>(blockIdx.x) * STRIP;
        const bool skip = SOFTMAX && causal && j_first > r_begin + m0 + TROWS - 1 + coff;
        // ... and one wholly before its columns' diagonal blocks stores nothing
        bool unstored = false;
        if constexpr (SOFTMAX) {
            const int64_t d = j_first - coff;
            const int64_t blk = d >= 0 ? d / 256 : -((-d + 255) / 256);
            unstored = causal && r_begin + m0 + TROWS - 1 < 256 * blk;
        }
#pragma unroll
        for (int r = 0; r < 8; ++r) {
            const uint32_t off = (col_off == kOut || skip) ? kOut
                               : static_cast<uint32_t>((m0 + 8 * mc + r) * ldx * 2) + col_off;
            const auto q = __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0);
            v[r] = make_uint4(q[0], q[1], q[2], q[3]);
        }
        if constexpr (NORM) {
#pragma unroll
            for (int r = 0; r < 8; ++r) {
                const int m = m0 + 8 * mc + r;
                const float sc = m < rows ? rsu[m] : 0.f;
                uint32_t w[4] = {v[r].x, v[r].y, v[r].z, v[r].w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float xa = __uint_as_float(w[e] << 16), xb = __uint_as_float(w[e] & 0xffff0000u);
                    w[e] = pack_bf16x2(bf16_to_f32(f32_to_bf16(xa * sc)) * gm[2 * e],
                                       bf16_to_f32(f32_to_bf16(xb * sc)) * gm[2 * e + 1]);
                }
                v[r] = make_uint4(w[0], w[1], w[2], w[3]);
            }
        }
        if constexpr (SOFTMAX) {
#pragma unroll
            for (int r = 0; r < 8; ++r) {
                const int m = m0 + 8 * mc + r;
                const bool live = m < rows;
                const float mx = live ? rsu[m] : 0.f, li = live ? riu[m] : 0.f;
                // keys j + e with j + e <= (r_begin + m) + coff are kept
                const int64_t lim = causal ? r_begin + m + coff - j : 8;
                uint32_t w[4] = {v[r].x, v[r].y, v[r].z, v[r].w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float sa = __uint_as_float(w[e] << 16), sb = __uint_as_float(w[e] & 0xffff0000u);
                    const float pa = (2 * e <= lim && li > 0.f) ? __expf(sa - mx) * li : 0.f;
                    const float pb = (2 * e + 1 <= lim && li > 0.f) ? __expf(sb - mx) * li : 0.f;
                    w[e] = pack_bf16x2(pa, pb);
                }
                v[r] = make_uint4(w[0], w[1], w[2], w[3]);
            }
        }
#pragma unroll
        for (int r = 0; r < 8; ++r) {
            const uint32_t w[4] = {v[r].x, v[r].y, v[r].z, v[r].w};
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const double x = e < nvalid
                    ? static_cast<double>(__uint_as_float((e & 1) ? (w[e >> 1] & 0xffff0000u) : (w[e >> 1] << 16)))
                    : 0.0;
                acc[e] = fma(x, x, acc[e]);
            }
        }
        if (XT && !unstored) {
            // column e of the 8 x 8 block becomes one 16-byte vector of Xt row j + e
            const int mrow = m0 + 8 * mc;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const uint32_t sel = (e & 1) ? 0x07060302u : 0x05040100u;
                uint32_t o[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const uint32_t a = reinterpret_cast<const uint32_t *>(&v[2 * q])[e >> 1];
                    const uint32_t b = reinterpret_cast<const uint32_t *>(&v[2 * q + 1])[e >> 1];
                    o[q] = __builtin_amdgcn_perm(b, a, sel);
                }
                if (e < nvalid) {
                    uint16_t *dst = xt + e * ldxt + mrow;
                    if (mrow + 8 <= rows) {
                        *reinterpret_cast<uint4 *>(dst) = make_uint4(o[0], o[1], o[2], o[3]);
                    } else {
#pragma unroll
                        for (int r = 0; r < 8; ++r)
                            if (mrow + r < rows) dst[r] = static_cast<uint16_t>(o[r >> 1] >> (16 * (r & 1)));
                    }
                }
            }
        }
    }
    // sum over the eight row groups of the wave (xor butterfly: every lane
    // ends with the same, order-independent sum), then over the waves in order
#pragma unroll
    for (int sh = JC; sh < 64; sh <<= 1)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] += __shfl_xor(acc[e], sh);
    if (mc == 0) {
#pragma unroll
        for (int e = 0; e < 8; ++e) red[wave][8 * jc + e] = acc[e];
    }
    __syncthreads();
    if (threadIdx.x < STRIP) {
        double s = red[0][threadIdx.x];
#pragma unroll
        for (int w = 1; w < kThreads / 64; ++w) s += red[w][threadIdx.x];
        const int64_t col = static_cast<int64_t>(blockIdx.x) * STRIP + threadIdx.x;
        if (col < K) out[unit * out_unit_stride + split * out_split_stride + col] = s;
    }
}

// energy[b][j] = sum over splits s (in order) of partials[b][s][j]
__global__ __launch_bounds__(64) void score_finalize_kernel(
    const double *__restrict__ partials, int64_t B, int64_t S, int64_t K,
    double *__restrict__ energy) {
    const int64_t t = static_cast<int64_t>(blockIdx.x) * 64 + threadIdx.x;
    if (t >= B * K) return;
    const int64_t b = t / K, j = t % K;
    const double *p = partials + b * S * K + j;
    double s = 0.0;
#pragma unroll 8
    for (int64_t i = 0; i < S; ++i) s += p[i * K];
    energy[t] = s;
}

// The same sum for many splits: 16 row groups of a column each add their
// ceil(S / 16) consecutive splits in order (16 loads in flight per thread),
// then the 16 group sums are added in group order.  64 columns per
// workgroup of 1024 threads.
constexpr int kFinGroups = 16;
__global__ __launch_bounds__(64 * kFinGroups) void score_finalize_grouped_kernel(
    const double *__restrict__ partials, int64_t S, int64_t K, double *__restrict__ energy) {
    const int c = threadIdx.x & 63, g = threadIdx.x >> 6;
    const int64_t j = static_cast<int64_t>(blockIdx.x) * 64 + c, b = blockIdx.y;
    const int64_t sg = (S + kFinGroups - 1) / kFinGroups;
    const int64_t s0 = g * sg, s1 = min(S, s0 + sg);
    double acc = 0.0;
    if (j < K) {
        const double *p = partials + b * S * K + j;
        int64_t s = s0;
        for (; s + 16 <= s1; s += 16) {
            double v[16];
#pragma unroll
            for (int i = 0; i < 16; ++i) v[i] = p[(s + i) * K];
#pragma unroll
            for (int i = 0; i < 16; ++i) acc += v[i];
        }
        for (; s < s1; ++s) acc += p[s * K];
    }
    __shared__ double red[kFinGroups][64];
    red[g][c] = acc;
    __syncthreads();
    if (g == 0 && j < K) {
        double t = red[0][c];
#pragma unroll
        for (int q = 1; q < kFinGroups; ++q) t += red[q][c];
        energy[b * K + j] = t;
    }
}

template <bool XT>
hipError_t launch_tiles(const uint16_t *X, int64_t B, int64_t M, int64_t K, int64_t ldx,
                        int64_t S, double *out, int64_t unit_stride, int64_t split_stride,
                        uint16_t *Xt, int64_t ldxt, hipStream_t stream) {
    const int64_t rps = score_rows_per_split(B, M, K);
    constexpr int strip = 8 * kTileJC;
    dim3 grid(static_cast<unsigned>((K + strip - 1) / strip), static_cast<unsigned>(S),
              static_cast<unsigned>(B));
    hipLaunchKernelGGL((score_tile_kernel<XT, kTileJC>), grid, dim3(kThreads), 0, stream, X, M, K,
                       ldx, rps, out, unit_stride, split_stride, Xt, ldxt);
    return hipGetLastError();
}

hipError_t launch_tiles_norm(const uint16_t *X, int64_t B, int64_t M, int64_t K, int64_t ldx,
                             int64_t S, double *out, int64_t unit_stride, int64_t split_stride,
                             uint16_t *Xt, int64_t ldxt, const float *rscale, const uint16_t *gamma,
                             hipStream_t stream) {
    const int64_t rps = score_rows_per_split(B, M, K);
    constexpr int strip = 8 * kTileJC;
    dim3 grid(static_cast<unsigned>((K + strip - 1) / strip), static_cast<unsigned>(S),
              static_cast<unsigned>(B));
    hipLaunchKernelGGL((score_tile_kernel<true, kTileJC, 1>), grid, dim3(kThreads), 0, stream, X, M,
                       K, ldx, rps, out, unit_stride, split_stride, Xt, ldxt, rscale, gamma);
    return hipGetLastError();
}

hipError_t launch_tiles_softmax(const uint16_t *S, int64_t B, int64_t M, int64_t K, int64_t ld,
                                int64_t splits, double *out, int64_t unit_stride, int64_t split_stride,
                                uint16_t *Pt, int64_t ldpt, const float *rmax, const float *rinv,
                                int64_t coff, int causal, hipStream_t stream) {
    const int64_t rps = score_rows_per_split(B, M, K);
    constexpr int strip = 8 * kTileJC;
    dim3 grid(static_cast<unsigned>((K + strip - 1) / strip), static_cast<unsigned>(splits),
              static_cast<unsigned>(B));
    hipLaunchKernelGGL((score_tile_kernel<true, kTileJC, 2>), grid, dim3(kThreads), 0, stream, S, M, K,
                       ld, rps, out, unit_stride, split_stride, Pt, ldpt, rmax, nullptr, rinv, coff,
                       causal);
    return hipGetLastError();
}

template <typename T, int VEC, bool XT>
hipError_t launch_partial(const T *X, int64_t B, int64_t M, int64_t K, int64_t ldx,
                          int64_t S, double *out, int64_t unit_stride, int64_t split_stride,
                          uint16_t *Xt, int64_t ldxt, hipStream_t stream) {
    const int64_t rps = score_rows_per_split(B, M, K);
    dim3 grid(static_cast<unsigned>((K + kScoreCols - 1) / kScoreCols),
              static_cast<unsigned>(S), static_cast<unsigned>(B));
    hipLaunchKernelGGL((score_partial_kernel<T, VEC, XT>), grid, dim3(kThreads), 0, stream,
                       X, M, K, ldx, rps, out, unit_stride, split_stride, Xt, ldxt);
    return hipGetLastError();
}

}  // namespace

// Rows per split: a whole number of 64-row slabs, chosen so that the grid
// of 64-column strips has about kScoreTargetBlocks workgroups.
int64_t score_rows_per_split(int64_t B, int64_t M, int64_t K) {
    const int64_t col_blocks = (K + kStrip - 1) / kStrip;
    int64_t s = (kScoreTargetBlocks + B * col_blocks - 1) / (B * col_blocks);
    const int64_t max_s = (M + kScoreMinRows - 1) / kScoreMinRows;
    if (s > max_s) s = max_s;
    if (s < 1) s = 1;
    int64_t rps = (M + s - 1) / s;
    rps = (rps + kScoreMinRows - 1) / kScoreMinRows * kScoreMinRows;
    if ((M + rps - 1) / rps > 65535) rps = (M + 65534) / 65535;
    return rps;
}

int64_t score_splits(int64_t B, int64_t M, int64_t K) {
    const int64_t rps = score_rows_per_split(B, M, K);
    return (M + rps - 1) / rps;
}

size_t score_workspace_bytes(int64_t B, int64_t M, int64_t K) {
    const int64_t s = score_splits(B, M, K);
    return s > 1 ? static_cast<size_t>(B * s * K) * sizeof(double) : 0;
}

hipError_t launch_score_norm_kmajor(const uint16_t *X, int64_t B, int64_t M, int64_t K, int64_t ldx,
                                   const float *rscale, const uint16_t *gamma, double *energy,
                                   double *partials, uint16_t *Xt, int64_t ldxt, hipStream_t stream) {
    const int64_t S = score_splits(B, M, K);
    double *out = S > 1 ? partials : energy;
    hipError_t err = launch_tiles_norm(X, B, M, K, ldx, S, out, S * K, K, Xt, ldxt, rscale, gamma,
                                       stream);
    if (err != hipSuccess || S == 1) return err;
    return launch_score_finalize(partials, B, S, K, energy, stream);
}

hipError_t launch_score_softmax_kmajor(const uint16_t *S, int64_t B, int64_t M, int64_t K, int64_t ld,
                                      const float *rmax, const float *rinv, int64_t coff,
                                      int causal, double *energy, double *partials, uint16_t *Pt,
                                      int64_t ldpt, hipStream_t stream) {
    const int64_t splits = score_splits(B, M, K);
    double *out = splits > 1 ? partials : energy;
    hipError_t err = launch_tiles_softmax(S, B, M, K, ld, splits, out, splits * K, K, Pt, ldpt, rmax,
                                          rinv, coff, causal, stream);
    if (err != hipSuccess || splits == 1) return err;
    return launch_score_finalize(partials, B, splits, K, energy, stream);
}

hipError_t launch_score_finalize(const double *partials, int64_t B, int64_t S, int64_t K,
                                 double *energy, hipStream_t stream) {
    const int64_t n = B * K;
    hipLaunchKernelGGL(score_finalize_kernel, dim3(static_cast<unsigned>((n + 63) / 64)), dim3(64), 0,
                       stream, partials, B, S, K, energy);
    return hipGetLastError();
}

hipError_t launch_score_finalize_grouped(const double *partials, int64_t B, int64_t S, int64_t K,
                                         double *energy, hipStream_t stream) {
    const dim3 grid(static_cast<unsigned>((K + 63) / 64), static_cast<unsigned>(B));
    hipLaunchKernelGGL(score_finalize_grouped_kernel, grid, dim3(64 * kFinGroups), 0, stream, partials,
                       S, K, energy);
    return hipGetLastError();
}

hipError_t launch_score(const void *X, bool bf16, int64_t B, int64_t M, int64_t K,
                        int64_t ldx, double *energy, double *partials, uint16_t *Xt,
                        int64_t ldxt, hipStream_t stream) {
    const int64_t S = score_splits(B, M, K);
    double *out = S > 1 ? partials : energy;
    const int64_t unit_stride = S * K, split_stride = K;
    const size_t esz = bf16 ? 2 : 4;
    const bool aligned = (reinterpret_cast<uintptr_t>(X) % 16 == 0) &&
                         ((ldx * static_cast<int64_t>(esz)) % 16 == 0);
    // the tile kernel addresses one split's rows with 32-bit byte offsets
    const bool tiles = bf16 && aligned &&
                       score_rows_per_split(B, M, K) * ldx * 2 < (int64_t(1) << 31);
    hipError_t err;
    if (Xt && tiles) {   // bf16, 16-byte aligned rows (checked by the caller)
        err = launch_tiles<true>(static_cast<const uint16_t *>(X), B, M, K, ldx, S, out, unit_stride,
                                 split_stride, Xt, ldxt, stream);
    } else if (Xt) {
        err = launch_partial<uint16_t, 8, true>(static_cast<const uint16_t *>(X), B, M, K, ldx, S, out,
                                                unit_stride, split_stride, Xt, ldxt, stream);
    } else if (bf16) {
        const uint16_t *x = static_cast<const uint16_t *>(X);
        err = tiles ? launch_tiles<false>(x, B, M, K, ldx, S, out, unit_stride, split_stride, nullptr,
                                          0, stream)
            : aligned ? launch_partial<uint16_t, 8, false>(x, B, M, K, ldx, S, out, unit_stride,
                                                           split_stride, nullptr, 0, stream)
                      : launch_partial<uint16_t, 1, false>(x, B, M, K, ldx, S, out, unit_stride,
                                                           split_stride, nullptr, 0, stream);
    } else {
        const float *x = static_cast<const float *>(X);
        err = aligned ? launch_partial<float, 4, false>(x, B, M, K, ldx, S, out, unit_stride,
                                                        split_stride, nullptr, 0, stream)
                      : launch_partial<float, 1, false>(x, B, M, K, ldx, S, out, unit_stride,
                                                        split_stride, nullptr, 0, stream);
    }
    if (err != hipSuccess || S == 1) return err;
    return launch_score_finalize(partials, B, S, K, energy, stream);
}

}  // namespace rmm
