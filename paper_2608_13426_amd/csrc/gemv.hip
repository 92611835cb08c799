// Reduced product with few rows per unit (a decode step: one token, or a
// handful, per sequence)   (Sec. 3.2 definition of RMM; App. A: during
// decoding the retained set follows the current decoding state).
//
//   Y[b][m][:] = sum_{t < k} X[b][m][I_b[t]] * W[I_b[t]][:],   m < M <= 8
//
// With so few rows the product is bound by reading the retained rows of W
// (k*N*2 bytes per unit): each retained index is one contiguous weight row,
// so the kernel streams exactly those rows.  Work is split over
// (512-column chunk, slice of the retained list, unit): a workgroup stages
// its slice's row offsets and activations in LDS, its four waves take every
// fourth row, each lane holding 8 columns (one 16-byte load per row, 8 rows
// in flight), and the waves' sums are added in a fixed order in LDS.  Slices write fp32 partials that a second kernel adds in slice
// order (or, with one slice, the workgroup writes Y directly), so results
// are bit-reproducible.
#include "device_common.h"
#include "kernels.h"

namespace rmm {

namespace {

namespace gv {
constexpr int NW = 4, NT = NW * 64;
constexpr int CW = 512;            // columns per workgroup (64 lanes x 8)
constexpr int RB = 256;            // retained rows staged per pass
constexpr int TARGET_BLOCKS = 512;
constexpr int MIN_SLICE = 64;      // retained rows per slice at least
}  // namespace gv

// One workgroup's share: columns chunk*CW .., slice s of unit b's retained
// list; DIRECT writes Y, otherwise the slice's fp32 partials.
template <int MR, bool VEC>
__device__ __forceinline__ void gemv_tile(
    const uint16_t *__restrict__ X, const uint16_t *__restrict__ W, const int32_t *__restrict__ idx,
    float *__restrict__ P, uint16_t *__restrict__ Y, int M, int N, int K, int k, int64_t ldx,
    int64_t ldw, int64_t ldy, int SR, int S, int chunk, int s, int b, bool DIRECT) {
    using namespace gv;
    __shared__ uint32_t roff[RB];              // byte offset of each staged row in W
    __shared__ float xs[RB][MR];               // its activation value per row m
    __shared__ float red[NW - 1][MR][CW];      // sums of waves 1..3

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n0 = chunk * CW;
    const int t0 = s * SR, t1 = min(k, t0 + SR);
    const int32_t *I = idx + static_cast<int64_t>(b) * k;
    const uint16_t *Xb = X + static_cast<int64_t>(b) * M * ldx;
    // the whole of W from this chunk's first column on: a row's columns past
    // N read padding or the next row, and past the matrix's end read zeros
    const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t *>(W + n0), 0,
        static_cast<uint32_t>((static_cast<int64_t>(K) * ldw - n0) * 2), 0x00020000);

    float acc[MR][8];
#pragma unroll
    for (int m = 0; m < MR; ++m)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[m][e] = 0.f;

    for (int base = t0; base < t1; base += RB) {
        const int nr = min(RB, t1 - base);
        for (int r = tid; r < nr; r += NT) {
            const int j = I[base + r];
            roff[r] = static_cast<uint32_t>(j * ldw * 2);
#pragma unroll
            for (int m = 0; m < MR; ++m)
                xs[r][m] = m < M ? bf16_to_f32(Xb[m * ldx + j]) : 0.f;
        }
        __syncthreads();
        // rows wave, wave + 4, ... of this pass; 8 loads in flight per lane
        for (int r0 = wave; r0 < nr; r0 += 8 * NW) {
            uint32_t w[8][4];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int r = r0 + NW * u;
                if (VEC) {
                    const uint32_t o = r < nr ? roff[r] + 16u * lane : 0x80000000u;
                    const auto v = __builtin_amdgcn_raw_buffer_load_b128(wr, o, 0, 0);
                    w[u][0] = v[0]; w[u][1] = v[1]; w[u][2] = v[2]; w[u][3] = v[3];
                } else {
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const uint32_t o = r < nr ? roff[r] + 16u * lane + 4u * q : 0x80000000u;
                        const uint32_t lo = __builtin_amdgcn_raw_buffer_load_b16(wr, o, 0, 0);
                        const uint32_t hi = __builtin_amdgcn_raw_buffer_load_b16(wr, o + 2u, 0, 0);
                        w[u][q] = lo | (hi << 16);
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int r = r0 + NW * u;
                if (r < nr) {
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const float wl = __uint_as_float(w[u][q] << 16);
                        const float wh = __uint_as_float(w[u][q] & 0xffff0000u);
#pragma unroll
                        for (int m = 0; m < MR; ++m) {
                            acc[m][2 * q] = __builtin_fmaf(xs[r][m], wl, acc[m][2 * q]);
                            acc[m][2 * q + 1] = __builtin_fmaf(xs[r][m], wh, acc[m][2 * q + 1]);
                        }
                    }
                }
            }
        }
        __syncthreads();                       // staged rows are reused by the next pass
    }

    // waves 1..3 hand their sums to wave 0, which adds them in wave order
    if (wave > 0) {
#pragma unroll
        for (int m = 0; m < MR; ++m)
#pragma unroll
            for (int e = 0; e < 8; ++e) red[wave - 1][m][8 * lane + e] = acc[m][e];
    }
    __syncthreads();
    if (wave != 0) return;
#pragma unroll
    for (int w = 0; w < NW - 1; ++w)
#pragma unroll
        for (int m = 0; m < MR; ++m)
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[m][e] += red[w][m][8 * lane + e];
    const int nb = n0 + 8 * lane;
#pragma unroll
    for (int m = 0; m < MR; ++m) {
        if (m >= M) break;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int n = nb + e;
            if (n < N) {
                if (DIRECT)
                    Y[(static_cast<int64_t>(b) * M + m) * ldy + n] = f32_to_bf16(acc[m][e]);
                else
                    P[((static_cast<int64_t>(b) * S + s) * M + m) * N + n] = acc[m][e];
            }
        }
    }
}

template <int MR, bool VEC, bool DIRECT>
__global__ __launch_bounds__(gv::NT) void gemv_partial_kernel(
    const uint16_t *__restrict__ X, const uint16_t *__restrict__ W, const int32_t *__restrict__ idx,
    float *__restrict__ P, uint16_t *__restrict__ Y, int M, int N, int K, int k, int64_t ldx,
    int64_t ldw, int64_t ldy, int SR, int S) {
    gemv_tile<MR, VEC>(X, W, idx, P, Y, M, N, K, k, ldx, ldw, ldy, SR, S, blockIdx.x, blockIdx.y,
                       blockIdx.z, DIRECT);
}

// Several independent one-row products in one launch: the workgroups of
// group g are g's (chunk, slice, unit) triples, numbered from first[g].
__global__ __launch_bounds__(gv::NT) void gemv_partial_grouped_kernel(GemvGroups G) {
    int g = 0;
    while (g + 1 < G.n && static_cast<int>(blockIdx.x) >= G.g[g + 1].first) ++g;
    const GemvGroup &q = G.g[g];
    const int local = static_cast<int>(blockIdx.x) - q.first;
    const int chunk = local % q.chunks, s = (local / q.chunks) % q.S, b = local / (q.chunks * q.S);
    gemv_tile<1, true>(q.X, q.W, q.idx, q.P, q.Y, 1, q.N, q.K, q.k, q.ldx, q.ldw, q.ldy, q.SR, q.S,
                       chunk, s, b, q.S == 1);
}

// The slice reduction of one 64-column piece: the 256 threads are 64
// columns (one per lane) x 4 waves; wave w adds slices [w*S/4, (w+1)*S/4)
// in slice order (eight loads in flight), and the four quarter sums are
// added in wave order.  p points at slice 0 of the lane's column; slice s
// is st floats further.  Returns the sum in wave 0 (other waves: garbage).
__device__ __forceinline__ float reduce_slices(const float *__restrict__ p, int64_t st, int S,
                                               bool col_ok) {
    __shared__ float quarter[3][64];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int s0 = w * S / 4, s1 = (w + 1) * S / 4;
    float sum = 0.f;
    if (col_ok) {
        int s = s0;
        for (; s + 8 <= s1; s += 8) {
            float v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = p[(s + u) * st];
#pragma unroll
            for (int u = 0; u < 8; ++u) sum += v[u];
        }
        for (; s < s1; ++s) sum += p[s * st];
    }
    if (w > 0) quarter[w - 1][lane] = sum;
    __syncthreads();
    if (w == 0) sum = ((sum + quarter[0][lane]) + quarter[1][lane]) + quarter[2][lane];
    return sum;
}

// Y[b][m][n] = the slices' partials P[b][s][m][n] added in the order of
// reduce_slices; workgroup (x, m, b) covers columns 64x .. 64x+63
__global__ __launch_bounds__(256) void gemv_reduce_kernel(const float *__restrict__ P,
                                                          uint16_t *__restrict__ Y, int M, int N,
                                                          int S, int64_t ldy) {
    const int n = blockIdx.x * 64 + (threadIdx.x & 63);
    const int m = blockIdx.y, b = blockIdx.z;
    const float *p = P + (static_cast<int64_t>(b) * S * M + m) * N + n;
    const float sum = reduce_slices(p, static_cast<int64_t>(M) * N, S, n < N);
    if (threadIdx.x < 64 && n < N) Y[(static_cast<int64_t>(b) * M + m) * ldy + n] = f32_to_bf16(sum);
}

// the slice reduction of every group with more than one slice: workgroup
// blockIdx.x of group g covers 64 columns of one unit, numbered from rfirst[g]
__global__ __launch_bounds__(256) void gemv_reduce_grouped_kernel(GemvGroups G) {
    int g = -1;
    for (int i = 0; i < G.n; ++i)
        if (G.g[i].S > 1 && static_cast<int>(blockIdx.x) >= G.g[i].rfirst) g = i;
    const GemvGroup &q = G.g[g];
    const int local = static_cast<int>(blockIdx.x) - q.rfirst;
    const int nb = (q.N + 63) / 64;
    const int b = local / nb, n = (local % nb) * 64 + static_cast<int>(threadIdx.x & 63);
    const float *p = q.P + static_cast<int64_t>(b) * q.S * q.N + n;
    const float sum = reduce_slices(p, q.N, q.S, n < q.N);
    if (threadIdx.x < 64 && n < q.N) q.Y[static_cast<int64_t>(b) * q.ldy + n] = f32_to_bf16(sum);
}

template <int MR, bool VEC>
hipError_t launch_mr(const uint16_t *X, const uint16_t *W, const int32_t *idx, int64_t B, int64_t M,
                     int64_t N, int64_t K, int64_t k, int64_t ldx, int64_t ldw, uint16_t *Y,
                     int64_t ldy, float *P, int SR, int S, hipStream_t stream) {
    using namespace gv;
    dim3 grid(static_cast<unsigned>((N + CW - 1) / CW), static_cast<unsigned>(S), static_cast<unsigned>(B));
    if (S == 1) {
        hipLaunchKernelGGL((gemv_partial_kernel<MR, VEC, true>), grid, dim3(NT), 0, stream, X, W, idx,
                           P, Y, static_cast<int>(M), static_cast<int>(N), static_cast<int>(K),
                           static_cast<int>(k), ldx, ldw, ldy, SR, S);
        return hipGetLastError();
    }
    hipLaunchKernelGGL((gemv_partial_kernel<MR, VEC, false>), grid, dim3(NT), 0, stream, X, W, idx,
                       P, Y, static_cast<int>(M), static_cast<int>(N), static_cast<int>(K),
                       static_cast<int>(k), ldx, ldw, ldy, SR, S);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    dim3 rgrid(static_cast<unsigned>((N + 63) / 64), static_cast<unsigned>(M), static_cast<unsigned>(B));
    hipLaunchKernelGGL(gemv_reduce_kernel, rgrid, dim3(256), 0, stream, P, Y, static_cast<int>(M),
                       static_cast<int>(N), S, ldy);
    return hipGetLastError();
}

template <bool VEC>
hipError_t launch_vec(const uint16_t *X, const uint16_t *W, const int32_t *idx, int64_t B, int64_t M,
                      int64_t N, int64_t K, int64_t k, int64_t ldx, int64_t ldw, uint16_t *Y,
                      int64_t ldy, float *P, int SR, int S, hipStream_t stream) {
    if (M == 1) return launch_mr<1, VEC>(X, W, idx, B, M, N, K, k, ldx, ldw, Y, ldy, P, SR, S, stream);
    if (M == 2) return launch_mr<2, VEC>(X, W, idx, B, M, N, K, k, ldx, ldw, Y, ldy, P, SR, S, stream);
    if (M <= 4) return launch_mr<4, VEC>(X, W, idx, B, M, N, K, k, ldx, ldw, Y, ldy, P, SR, S, stream);
    return launch_mr<8, VEC>(X, W, idx, B, M, N, K, k, ldx, ldw, Y, ldy, P, SR, S, stream);
}

}  // namespace

// Rows per slice (a multiple of 4) and slice count: enough workgroups to
// keep every CU streaming, at least MIN_SLICE rows per slice.
void gemv_slices(int64_t B, int64_t N, int64_t k, int *SR, int *S) {
    const int64_t chunks = (N + gv::CW - 1) / gv::CW;
    int64_t s = (gv::TARGET_BLOCKS + B * chunks - 1) / (B * chunks);
    const int64_t smax = (k + gv::MIN_SLICE - 1) / gv::MIN_SLICE;
    if (s > smax) s = smax;
    if (s < 1) s = 1;
    int64_t sr = (k + s - 1) / s;
    sr = (sr + 3) / 4 * 4;
    *SR = static_cast<int>(sr);
    *S = static_cast<int>((k + sr - 1) / sr);
}

size_t gemv_workspace_bytes(int64_t B, int64_t M, int64_t N, int64_t k) {
    int SR, S;
    gemv_slices(B, N, k, &SR, &S);
    return S == 1 ? 0 : static_cast<size_t>(B) * S * M * N * sizeof(float);
}

hipError_t launch_gemv_grouped_bf16(GemvGroups G, int64_t B, hipStream_t stream) {
    int blocks = 0, rblocks = 0;
    for (int i = 0; i < G.n; ++i) {
        GemvGroup &q = G.g[i];
        gemv_slices(B, q.N, q.k, &q.SR, &q.S);
        q.chunks = (q.N + gv::CW - 1) / gv::CW;
        q.first = blocks;
        blocks += q.chunks * q.S * static_cast<int>(B);
        q.rfirst = rblocks;
        if (q.S > 1) rblocks += (q.N + 63) / 64 * static_cast<int>(B);
    }
    hipLaunchKernelGGL(gemv_partial_grouped_kernel, dim3(static_cast<unsigned>(blocks)), dim3(gv::NT), 0,
                       stream, G);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || rblocks == 0) return e;
    hipLaunchKernelGGL(gemv_reduce_grouped_kernel, dim3(static_cast<unsigned>(rblocks)), dim3(256), 0,
                       stream, G);
    return hipGetLastError();
}

hipError_t launch_gemv_bf16(const uint16_t *X, const uint16_t *W, const int32_t *idx, int64_t B,
                            int64_t M, int64_t N, int64_t K, int64_t k, int64_t ldx, int64_t ldw,
                            uint16_t *Y, int64_t ldy, void *workspace, hipStream_t stream) {
    int SR, S;
    gemv_slices(B, N, k, &SR, &S);
    const bool vec = ldw % 8 == 0 && reinterpret_cast<uintptr_t>(W) % 16 == 0;
    float *P = static_cast<float *>(workspace);
    return vec ? launch_vec<true>(X, W, idx, B, M, N, K, k, ldx, ldw, Y, ldy, P, SR, S, stream)
               : launch_vec<false>(X, W, idx, B, M, N, K, k, ldx, ldw, Y, ldy, P, SR, S, stream);
}

}  // namespace rmm
