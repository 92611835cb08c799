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
#include <type_traits>

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

// ------------------------------------------------------ bf16, large tiles
// 256x256 output tile, 64 retained indices per k-tile, NW waves in a 2 x NW/2
// grid (each wave 128 x 512/NW), LDS double-buffered (128 KB).  Each LDS row
// holds the 64 k-values of one output row (A) or column (B) as eight 16-byte
// chunks; chunk c of row r is stored at c ^ swz(r), which spreads the operand
// reads of 8 consecutive rows, the gathered-X writes and the transposed-W
// writes of rows 8 apart over distinct bank groups.
namespace big {
constexpr int BM = 256, BN = 256, BK = 64;
constexpr int GROUP_M = 4;
__device__ __forceinline__ int swz(int row) { return (row ^ (row >> 3)) & 7; }
__device__ __forceinline__ int at(int row, int chunk) { return row * BK + ((chunk ^ swz(row)) << 3); }
}  // namespace big

template <int NW>
__global__ __launch_bounds__(NW * 64, NW / 4) void gemm_gather_bf16_big_kernel(
    const uint16_t *__restrict__ X, const uint16_t *__restrict__ W,
    const int32_t *__restrict__ idx, uint16_t *__restrict__ Y, int M, int N, int k,
    int64_t ldx, int64_t ldw, int64_t ldy, int64_t w_bytes, int tiles_m, int tiles_n) {
    using namespace big;
    constexpr int NT = NW * 64;
    constexpr int WN = NW / 2;            // waves along N (2 along M)
    constexpr int TN = BN / WN;           // wave tile: 128 x TN
    constexpr int FN = TN / 32;
    constexpr int XR = BM / (2 * NW);     // X rows gathered per thread (pairs)
    constexpr int WR = BK * BN / 8 / NT;  // W rows per thread block (8 columns wide)
    static_assert(WR == 4 || WR == 8, "W block");
    __shared__ __attribute__((aligned(16))) uint16_t lds[2 * (BM + BN) * BK];
    // buffer b: A tile at lds + b*BM*BK, B tile at lds + 2*BM*BK + b*BN*BK

    // XCD-aware raster: workgroups are dealt round-robin to the 8 XCDs, so
    // give each XCD one contiguous run of tiles, ordered GROUP_M rows of
    // tiles at a time, so that the XCD's L2 serves shared X and W panels.
    const int T = tiles_m * tiles_n;
    const int bid = blockIdx.x;
    const int lin = (T % 8 == 0) ? (bid % 8) * (T / 8) + bid / 8 : bid;
    const int gsz = GROUP_M * tiles_n;
    const int first_m = (lin / gsz) * GROUP_M;
    const int gm = min(GROUP_M, tiles_m - first_m);
    const int m0 = (first_m + (lin % gsz) % gm) * BM;
    const int n0 = ((lin % gsz) / gm) * BN;
    const int64_t unit = blockIdx.y;
    X += unit * static_cast<int64_t>(M) * ldx;
    Y += unit * static_cast<int64_t>(M) * ldy;
    idx += unit * k;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // X gather: lane pair p takes retained positions 2p, 2p+1 of rows ra + 2*NW*i
    const int p = lane & 31, ra = wave * 2 + (lane >> 5);
    // W gather: a WR x 8 block, rows WR*tq.. of the k-tile, columns 8*c..
    const int tq = tid >> 5, c = tid & 31;

    uint32_t xlo[XR], xhi[XR];
    uint4 wv[WR];

    // Branch-free gathers through buffer descriptors: a lane whose retained
    // position is past k, or whose row is past M, reads at an offset beyond
    // the descriptor's range and gets zero from the hardware.  Columns past
    // N read neighbouring data that only reaches outputs that are never
    // stored.  Byte offsets fit 31 bits (checked by the launcher).
    constexpr uint32_t kOut = 0x80000000u;
    const uint32_t xrow = static_cast<uint32_t>(ldx) * 2u;
    const uint32_t x_bytes = static_cast<uint32_t>(min(M - m0, BM)) * xrow;
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t *>(X + static_cast<int64_t>(m0) * ldx), 0, x_bytes, 0x00020000);
    const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t *>(W), 0, static_cast<uint32_t>(w_bytes), 0x00020000);
    const __amdgpu_buffer_rsrc_t ir = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int32_t *>(idx), 0, static_cast<uint32_t>(k) * 4u, 0x00020000);
    const uint32_t xlane = static_cast<uint32_t>(ra) * xrow;
    const uint32_t wcol = static_cast<uint32_t>(n0 + 8 * c) * 2u;
    const uint32_t wrow = static_cast<uint32_t>(ldw) * 2u;

    // Index values are fetched one k-tile ahead of the gathers that use them
    // (raw[]), then turned into byte offsets (off[]) once they have landed.
    uint32_t raw[2 + WR], off[2 + WR];
    auto fetch_idx = [&](int t0) {
        raw[0] = __builtin_amdgcn_raw_buffer_load_b32(ir, static_cast<uint32_t>(t0 + 2 * p) * 4u, 0, 0);
        raw[1] = __builtin_amdgcn_raw_buffer_load_b32(ir, static_cast<uint32_t>(t0 + 2 * p + 1) * 4u, 0, 0);
#pragma unroll
        for (int i = 0; i < WR; ++i)
            raw[2 + i] = __builtin_amdgcn_raw_buffer_load_b32(
                ir, static_cast<uint32_t>(t0 + WR * tq + i) * 4u, 0, 0);
    };
    auto make_offsets = [&](int t0) {
        off[0] = t0 + 2 * p < k ? raw[0] * 2u : kOut;
        off[1] = t0 + 2 * p + 1 < k ? raw[1] * 2u : kOut;
#pragma unroll
        for (int i = 0; i < WR; ++i) off[2 + i] = t0 + WR * tq + i < k ? raw[2 + i] * wrow + wcol : kOut;
    };
    auto gather = [&]() {
#pragma unroll
        for (int i = 0; i < XR; ++i) {
            const uint32_t row = xlane + static_cast<uint32_t>(2 * NW * i) * xrow;
            // packed into pairs only at stash time, so no wait sits between loads
            xlo[i] = __builtin_amdgcn_raw_buffer_load_b16(xr, row + off[0], 0, 0);
            xhi[i] = __builtin_amdgcn_raw_buffer_load_b16(xr, row + off[1], 0, 0);
        }
#pragma unroll
        for (int i = 0; i < WR; ++i) {
            const auto v = __builtin_amdgcn_raw_buffer_load_b128(wr, off[2 + i], 0, 0);
            wv[i] = make_uint4(v[0], v[1], v[2], v[3]);
        }
    };
    auto stash = [&](uint16_t *as, uint16_t *bs) {
#pragma unroll
        for (int i = 0; i < XR; ++i) {
            const int row = ra + 2 * NW * i;
            *reinterpret_cast<uint32_t *>(&as[at(row, p >> 2) + 2 * (p & 3)]) = xlo[i] | (xhi[i] << 16);
        }
        // WR x 8 transpose: column jj of the block becomes WR consecutive k of B row n
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) {
            uint32_t d[WR / 2];
#pragma unroll
            for (int q = 0; q < WR / 2; ++q) {
                const uint32_t a = reinterpret_cast<const uint32_t *>(&wv[2 * q])[jj >> 1];
                const uint32_t b = reinterpret_cast<const uint32_t *>(&wv[2 * q + 1])[jj >> 1];
                d[q] = (jj & 1) ? ((a >> 16) | (b & 0xffff0000u)) : ((a & 0xffffu) | (b << 16));
            }
            if constexpr (WR == 8) {
                *reinterpret_cast<uint4 *>(&bs[at(8 * c + jj, tq)]) = make_uint4(d[0], d[1], d[2], d[3]);
            } else {
                *reinterpret_cast<uint2 *>(&bs[at(8 * c + jj, tq >> 1) + 4 * (tq & 1)]) = make_uint2(d[0], d[1]);
            }
        }
    };

    f32x16_t acc[4][FN];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    const int wm = wave / WN, wn = wave % WN;
    const int lr = lane & 31, lh = lane >> 5;
    const int nT = (k + BK - 1) / BK;
    fetch_idx(0);
    make_offsets(0);
    gather();
    if (nT > 1) fetch_idx(BK);
    stash(lds, lds + 2 * BM * BK);
    if (nT > 1) make_offsets(BK);
    __syncthreads();
    for (int t = 0; t < nT; ++t) {
        const int cur = t & 1;
        const uint16_t *as = lds + cur * BM * BK;
        const uint16_t *bs = lds + 2 * BM * BK + cur * BN * BK;
        if (t + 2 < nT) fetch_idx((t + 2) * BK);
        if (t + 1 < nT) gather();
#pragma unroll
        for (int ks = 0; ks < BK / 16; ++ks) {
            const int chunk = 2 * ks + lh;
            bf16x8_t a[4], b[FN];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                a[i] = *reinterpret_cast<const bf16x8_t *>(&as[at(wm * 128 + i * 32 + lr, chunk)]);
#pragma unroll
            for (int j = 0; j < FN; ++j)
                b[j] = *reinterpret_cast<const bf16x8_t *>(&bs[at(wn * TN + j * 32 + lr, chunk)]);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
        }
        if (t + 1 < nT) stash(lds + (cur ^ 1) * BM * BK, lds + 2 * BM * BK + (cur ^ 1) * BN * BK);
        if (t + 2 < nT) make_offsets((t + 2) * BK);
        __syncthreads();
    }

#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const int n = n0 + wn * TN + j * 32 + lr;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int m = m0 + wm * 128 + i * 32 + 8 * (v / 4) + 4 * lh + (v % 4);
                if (m < M && n < N) Y[static_cast<int64_t>(m) * ldy + n] = f32_to_bf16(acc[i][j][v]);
            }
        }
}

// ------------------------------------------- bf16, K-major activations
// Xt[j][m] holds X[m][j] (written by the scoring pass), so a retained index
// is one contiguous row of Xt, just as it is one contiguous row of W.  Both
// operands are gathered as 16-byte row vectors: each thread loads an R x 8
// block (R retained rows, 8 consecutive m or n), transposes it in registers
// and writes 8 LDS rows of R consecutive k -- the swizzled layout of the
// large-tile kernel above.  Square tiles of BT = 256 (four waves of 128x128)
// or 128 (four waves of 64x64); 64 retained indices per k-tile.
template <int BT, int NW>
__global__ __launch_bounds__(NW * 64, NW / 4) void gemm_kmajor_bf16_kernel(
    const uint16_t *__restrict__ Xt, const uint16_t *__restrict__ W,
    const int32_t *__restrict__ idx, uint16_t *__restrict__ Y, int M, int N, int K, int k,
    int64_t ldxt, int64_t ldw, int64_t ldy, int64_t xt_bytes, int64_t w_bytes, int tiles_m,
    int tiles_n) {
    using big::at;
    constexpr int BK = big::BK, NT = NW * 64;
    constexpr int G = BT / 8;             // 8-wide column groups per tile row
    constexpr int R = BK * G / NT;        // retained rows per thread block
    constexpr int WN = NW / 2;            // waves: 2 along M, NW/2 along N
    constexpr int TWM = BT / 2, TWN = BT / WN;
    constexpr int FM = TWM / 32, FN = TWN / 32;
    static_assert(R == 4 || R == 8, "thread block");
    __shared__ __attribute__((aligned(16))) uint16_t lds[2 * 2 * BT * BK];

    const int T = tiles_m * tiles_n;
    const int bid = blockIdx.x;
    const int lin = (T % 8 == 0) ? (bid % 8) * (T / 8) + bid / 8 : bid;
    const int gsz = big::GROUP_M * tiles_n;
    const int first_m = (lin / gsz) * big::GROUP_M;
    const int gm = min(big::GROUP_M, tiles_m - first_m);
    const int m0 = (first_m + (lin % gsz) % gm) * BT;
    const int n0 = ((lin % gsz) / gm) * BT;
    const int64_t unit = blockIdx.y;
    Xt += unit * static_cast<int64_t>(K) * ldxt;
    Y += unit * static_cast<int64_t>(M) * ldy;
    idx += unit * k;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int c = tid % G, tq = tid / G;   // columns 8c.., retained rows R*tq..

    // Rows past k read out of range (zero); columns past M or N read
    // neighbouring data that only reaches outputs never stored.
    constexpr uint32_t kOut = 0x80000000u;
    const __amdgpu_buffer_rsrc_t ar = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t *>(Xt), 0, static_cast<uint32_t>(xt_bytes), 0x00020000);
    const __amdgpu_buffer_rsrc_t br = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t *>(W), 0, static_cast<uint32_t>(w_bytes), 0x00020000);
    const __amdgpu_buffer_rsrc_t ir = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int32_t *>(idx), 0, static_cast<uint32_t>(k) * 4u, 0x00020000);
    const uint32_t arow = static_cast<uint32_t>(ldxt) * 2u, brow = static_cast<uint32_t>(ldw) * 2u;
    const uint32_t acol = static_cast<uint32_t>(m0 + 8 * c) * 2u;
    const uint32_t bcol = static_cast<uint32_t>(n0 + 8 * c) * 2u;

    uint32_t raw[R], ao[R], bo[R];
    uint4 av[R], bv[R];
    auto fetch_idx = [&](int t0) {
#pragma unroll
        for (int i = 0; i < R; ++i)
            raw[i] = __builtin_amdgcn_raw_buffer_load_b32(ir, static_cast<uint32_t>(t0 + R * tq + i) * 4u, 0, 0);
    };
    auto make_offsets = [&](int t0) {
#pragma unroll
        for (int i = 0; i < R; ++i) {
            const bool in = t0 + R * tq + i < k;
            ao[i] = in ? raw[i] * arow + acol : kOut;
            bo[i] = in ? raw[i] * brow + bcol : kOut;
        }
    };
    auto gather = [&]() {
#pragma unroll
        for (int i = 0; i < R; ++i) {
            const auto a = __builtin_amdgcn_raw_buffer_load_b128(ar, ao[i], 0, 0);
            av[i] = make_uint4(a[0], a[1], a[2], a[3]);
        }
#pragma unroll
        for (int i = 0; i < R; ++i) {
            const auto b = __builtin_amdgcn_raw_buffer_load_b128(br, bo[i], 0, 0);
            bv[i] = make_uint4(b[0], b[1], b[2], b[3]);
        }
    };
    // R x 8 block -> 8 LDS rows (8c + jj) of R consecutive k
    auto put = [&](uint16_t *dst, const uint4 *v) {
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) {
            uint32_t d[R / 2];
#pragma unroll
            for (int q = 0; q < R / 2; ++q) {
                const uint32_t a = reinterpret_cast<const uint32_t *>(&v[2 * q])[jj >> 1];
                const uint32_t b = reinterpret_cast<const uint32_t *>(&v[2 * q + 1])[jj >> 1];
                d[q] = (jj & 1) ? ((a >> 16) | (b & 0xffff0000u)) : ((a & 0xffffu) | (b << 16));
            }
            if constexpr (R == 8)
                *reinterpret_cast<uint4 *>(&dst[at(8 * c + jj, tq)]) = make_uint4(d[0], d[1], d[2], d[3]);
            else
                *reinterpret_cast<uint2 *>(&dst[at(8 * c + jj, tq >> 1) + 4 * (tq & 1)]) = make_uint2(d[0], d[1]);
        }
    };

    f32x16_t acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    const int wm = wave / WN, wn = wave % WN;
    const int lr = lane & 31, lh = lane >> 5;
    const int nT = (k + BK - 1) / BK;
    // buffer b: A at lds + b*BT*BK, B at lds + (2 + b)*BT*BK
    fetch_idx(0);
    make_offsets(0);
    gather();
    if (nT > 1) fetch_idx(BK);
    put(lds, av);
    put(lds + 2 * BT * BK, bv);
    if (nT > 1) make_offsets(BK);
    __syncthreads();
    for (int t = 0; t < nT; ++t) {
        const int cur = t & 1;
        const uint16_t *as = lds + cur * BT * BK;
        const uint16_t *bs = lds + (2 + cur) * BT * BK;
        if (t + 2 < nT) fetch_idx((t + 2) * BK);
        if (t + 1 < nT) gather();
#pragma unroll
        for (int ks = 0; ks < BK / 16; ++ks) {
            const int chunk = 2 * ks + lh;
            bf16x8_t a[FM], b[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i)
                a[i] = *reinterpret_cast<const bf16x8_t *>(&as[at(wm * TWM + i * 32 + lr, chunk)]);
#pragma unroll
            for (int j = 0; j < FN; ++j)
                b[j] = *reinterpret_cast<const bf16x8_t *>(&bs[at(wn * TWN + j * 32 + lr, chunk)]);
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
        }
        if (t + 1 < nT) {
            put(lds + (cur ^ 1) * BT * BK, av);
            put(lds + (2 + (cur ^ 1)) * BT * BK, bv);
        }
        if (t + 2 < nT) make_offsets((t + 2) * BK);
        __syncthreads();
    }

#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const int n = n0 + wn * TWN + j * 32 + lr;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int m = m0 + wm * TWM + i * 32 + 8 * (v / 4) + 4 * lh + (v % 4);
                if (m < M && n < N) Y[static_cast<int64_t>(m) * ldy + n] = f32_to_bf16(acc[i][j][v]);
            }
        }
}

// ---------------------- bf16, K-major activations, DMA + transposing reads
// Same operands as above (rows I(t) of Xt and of W), but nothing passes
// through registers on the way in: each wave issues 16-byte buffer loads
// that land directly in LDS (a wave fills 1 KiB = two 512-byte staged rows
// of one operand), and the MFMA fragments are read back with the gfx950
// transposing LDS read, which hands each lane four consecutive k of one m
// (or n) from a K-major tile.  Within a staged row the 16-byte chunk c is
// stored at position c ^ 4*(row % 4), so that the four rows one 16-lane
// group reads together land in distinct banks.  Retained rows past k read
// out of range and stage zeros.
//
// The K loop is a ring of S stages of BKS retained rows; loads run S-1
// stages ahead of the MFMAs, so a gather has S-1 stage times to arrive.  The
// retained indices are read with scalar loads (a wave's rows are
// contiguous in the index list), which keeps them off the vector-memory
// counter: waiting for the stage about to be consumed never waits for the
// younger stages still in flight.
//
// The product is formed as Y^T tiles (W fragment as the MFMA's first
// operand), so each lane ends with four consecutive n of one m and stores
// them as one 8-byte vector.
namespace trk {
constexpr int BT = 256;
constexpr int ROWB = BT * 2;             // bytes per staged row
// s_waitcnt vmcnt(N) with expcnt and lgkmcnt unconstrained
template <int N>
__device__ __forceinline__ void wait_vmcnt_le() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
}
}  // namespace trk

// bf16(bf16(silu(g)) * u) for bf16 g, u (bits in the low half); silu(g) =
// g / (1 + e^-g) in fp32 with the hardware exp2 and reciprocal (each about
// one ulp), far below the bf16 rounding that follows
__device__ __forceinline__ uint32_t swiglu_bf16(uint32_t gb, uint32_t ub) {
    const float g = __uint_as_float(gb << 16), u = __uint_as_float(ub << 16);
    const float sg = bf16_to_f32(f32_to_bf16(g * __builtin_amdgcn_rcpf(1.f + __expf(-g))));
    return f32_to_bf16(sg * u);
}

// EPI selects the epilogue.  0: Y = the product.  1 (SwiGLU): the weight
// columns come in 128-column blocks, gate then up of the same 128 channels,
// so a 256-column tile holds both halves of channels c0 = n0/2 .. c0+127;
// the tile writes, for the down projection that follows,
//   Ht[unit][c][m] = bf16(bf16(silu(g[m][c])) * u[m][c])   (K-major, row
//   stride ldy; g and u the bf16-rounded products, as a plain launch would
//   store them),
// and part[(unit * tiles_m + m0/256) * N/2 + c] = sum over its rows m < M of
// Ht[unit][c][m]^2 in float64 (one row tile's share of that input's column
// energies).
//
// BNT is the tile's width in n: 256 (eight waves, one workgroup per CU), or
// 128 (four waves of the same 128 x 64 wave tile, 72 KiB of LDS, two
// workgroups per CU whose barriers and epilogues need not coincide).  With
// BNT = 128 a staged W row is 256 bytes and one wave instruction stages four
// of them.  OCC is the waves per SIMD the register budget is sized for.
template <int NW, int BKS, int S, int EPI = 0, int BNT = 256, int OCC = NW / 4>
__global__ __launch_bounds__(NW * 64, OCC) void gemm_kmajor_tr_kernel(
    const uint16_t *__restrict__ Xt, const uint16_t *__restrict__ W,
    const int32_t *__restrict__ idx, uint16_t *__restrict__ Y, int M, int N, int k,
    int64_t ldxt, int64_t ldw, int64_t ldy, int64_t xt_bytes, int64_t w_bytes, int tiles_m,
    int tiles_n, int vec_y, double *__restrict__ part, int64_t w_ustride = 0, int w_ugroup = 1,
    int trim = 0, int64_t trim_off = 0) {
    using namespace trk;
    constexpr int ASZ = BKS * ROWB;      // X operand, one stage
    constexpr int ROWBB = BNT * 2;       // bytes per staged W row
    constexpr int BSZ = BKS * ROWBB;     // W operand, one stage
    constexpr int PPW = BKS / 2 / NW;    // staged X row pairs per wave
    constexpr int RPB = 1024 / ROWBB;    // W rows one wave instruction stages
    constexpr int BLD = BKS / RPB / NW;  // W loads per wave per stage
    constexpr int WN = NW / 2;           // waves: 2 along m, NW/2 along n
    constexpr int TWN = BNT / WN;
    constexpr int FM = 4, FN = TWN / 32;
    constexpr int D = S - 1;             // stages in flight ahead of the MFMAs
    constexpr int PER_STAGE = PPW + BLD; // loads per wave per stage
    static_assert((NW == 4 || NW == 8) && PPW * NW * 2 == BKS && PPW >= 1, "wave layout");
    static_assert((BNT == 256 || BNT == 128) && BLD * RPB * NW == BKS && BLD >= 1 && FN >= 1,
                  "W staging layout");
    static_assert(BKS % 16 == 0 && S >= 2 && S <= 4 && S * (ASZ + BSZ) <= 160 * 1024, "stages");
    static_assert((D - 1) * PER_STAGE < 64, "vmcnt range");
    // One LDS object per stage and operand: the compiler then sees that a
    // fragment read of one stage cannot alias the loads still landing in the
    // others, and waits only for the loads of the stage it reads.
    __shared__ __attribute__((aligned(1024))) char sA0[ASZ], sA1[ASZ], sA2[ASZ], sA3[ASZ];
    __shared__ __attribute__((aligned(1024))) char sB0[BSZ], sB1[BSZ], sB2[BSZ], sB3[BSZ];
    auto stage_a = [&](auto I) -> char * {
        constexpr int i = decltype(I)::value;
        if constexpr (i == 0) return sA0;
        else if constexpr (i == 1) return sA1;
        else if constexpr (i == 2) return sA2;
        else return sA3;
    };
    auto stage_b = [&](auto I) -> char * {
        constexpr int i = decltype(I)::value;
        if constexpr (i == 0) return sB0;
        else if constexpr (i == 1) return sB1;
        else if constexpr (i == 2) return sB2;
        else return sB3;
    };

    const int T = tiles_m * tiles_n;
    const int bid = blockIdx.x;
    const int lin = (T % 8 == 0) ? (bid % 8) * (T / 8) + bid / 8 : bid;
    const int gsz = big::GROUP_M * tiles_n;
    const int first_m = (lin / gsz) * big::GROUP_M;
    const int gm = min(big::GROUP_M, tiles_m - first_m);
    const int m0 = (first_m + (lin % gsz) % gm) * BT;
    const int n0 = ((lin % gsz) / gm) * BNT;
    const int64_t unit = blockIdx.y;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int32_t *I = idx + unit * k;
    // trim: X is zero at (m, j) for j > m + trim_off (a causal operand), so
    // the retained indices past this tile's last row's limit add nothing and
    // the K loop stops before them (I is ascending: a binary search)
    int kk = k;
    if (trim) {
        const int64_t jmax = static_cast<int64_t>(m0) + BT - 1 + trim_off;
        int lo = 0, hi = k;
        while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            if (static_cast<int64_t>(I[mid]) <= jmax) lo = mid + 1; else hi = mid;
        }
        kk = __builtin_amdgcn_readfirstlane(lo);
    }

    constexpr uint32_t kOut = 0x80000000u;
    const __amdgpu_buffer_rsrc_t ar = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t *>(Xt + unit * (xt_bytes / 2)), 0, static_cast<uint32_t>(xt_bytes),
        0x00020000);
    // units u read weights W + (u / w_ugroup) * w_ustride (one matrix for all
    // units unless the caller groups them, e.g. query heads sharing a value head)
    const __amdgpu_buffer_rsrc_t br = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t *>(W + (unit / w_ugroup) * w_ustride), 0, static_cast<uint32_t>(w_bytes),
        0x00020000);
    const uint32_t arow = static_cast<uint32_t>(ldxt) * 2u, brow = static_cast<uint32_t>(ldw) * 2u;

    // DMA role: row pair P = wave*PPW + q of a stage holds retained rows
    // 2P + h; this lane fills chunk position p of its row with source chunk
    // p ^ 4*(row % 4), and row % 4 = (2P + h) % 4.
    const int h = lane >> 5, p = lane & 31;
    uint32_t acol[2], bcol[2];
#pragma unroll
    for (int e = 0; e < 2; ++e) {
        const int src = p ^ (4 * ((2 * e + h) & 3));
        acol[e] = static_cast<uint32_t>(m0 + 8 * src) * 2u;
        bcol[e] = static_cast<uint32_t>(n0 + 8 * src) * 2u;
    }
    // BNT = 128: lane l fills chunk position l % 16 of staged W row l / 16 of
    // its instruction's four, with source chunk (l % 16) ^ 4*(row % 4)
    const int bq = lane >> 4;
    const uint32_t bcol4 = static_cast<uint32_t>(n0 + 8 * ((lane & 15) ^ (4 * bq))) * 2u;
    // the wave's 2*PPW retained positions of stage st, read as scalars
    // (clamped into the list; positions past k are masked below)
    auto stage_idx = [&](int st, int32_t (&r)[2 * PPW]) {
        const int base = st * BKS + 2 * wave * PPW;
#pragma unroll
        for (int e = 0; e < 2 * PPW; ++e) r[e] = I[min(base + e, k - 1)];   // positions >= kk: masked
    };
    auto dma = [&](auto slot, int st, const int32_t (&r)[2 * PPW]) {
        char *la = stage_a(slot), *lb = stage_b(slot);
        const int base = st * BKS + 2 * wave * PPW;
#pragma unroll
        for (int q = 0; q < PPW; ++q) {
            const bool in = base + 2 * q + h < kk;
            const uint32_t j = static_cast<uint32_t>(h ? r[2 * q + 1] : r[2 * q]);
            const int P = wave * PPW + q;
            const uint32_t ao = in ? j * arow + acol[P & 1] : kOut;
            lds_load16(ar, la + P * 1024, ao);
            if constexpr (BNT == 256) {
                const uint32_t bo = in ? j * brow + bcol[P & 1] : kOut;
                lds_load16(br, lb + P * 1024, bo);
            }
        }
        if constexpr (BNT == 128) {
#pragma unroll
            for (int q = 0; q < BLD; ++q) {
                const int local = RPB * q + bq;           // row within the wave's 2*PPW
                const bool in = base + local < kk;
                uint32_t j = static_cast<uint32_t>(r[0]);
#pragma unroll
                for (int e = 1; e < 2 * PPW; ++e)
                    if (local == e) j = static_cast<uint32_t>(r[e]);
                const uint32_t bo = in ? j * brow + bcol4 : kOut;
                lds_load16(br, lb + (wave * BLD + q) * 1024, bo);
            }
        }
    };

    // Fragment role: 16-lane group g reads rows 8*(g/2) + s/4 (+4) of a
    // 16-row k-step, columns 16*(g%2) + 4*(s%4) .. +3 of a 32-wide block.
    const int wm = wave / WN, wn = wave % WN;
    const int g = lane >> 4, s16 = lane & 15;
    const int f4 = (s16 >> 2) & 3;
    const int col_off = (2 * (g & 1) + ((s16 & 3) >> 1)) * 16 + 8 * (s16 & 1);
    const int lane_off = (8 * (g >> 1) + (s16 >> 2)) * ROWB + col_off;
    const int lane_off_b = (8 * (g >> 1) + (s16 >> 2)) * ROWBB + col_off;
    int aoff[FM], boff[FN];
#pragma unroll
    for (int i = 0; i < FM; ++i) aoff[i] = lane_off + 64 * (4 * wm + (i ^ f4));
#pragma unroll
    for (int j = 0; j < FN; ++j) {
        const int q = (wn * TWN) / 32 + j;
        boff[j] = lane_off_b + 64 * ((q & ~3) + ((q & 3) ^ f4));
    }
    auto frag = [&](const char *base, auto RB) -> bf16x8_t {
        constexpr int rb = decltype(RB)::value;
        const s16x4_t lo = lds_read_tr16(base);
        const s16x4_t hi = lds_read_tr16(base + 4 * rb);
        typedef short s16x8_t __attribute__((ext_vector_type(8)));
        const s16x8_t v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        return __builtin_bit_cast(bf16x8_t, v);
    };

    f32x16_t acc[FN][FM];
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[j][i][v] = 0.f;

    const int nT = (kk + BKS - 1) / BKS;
    int32_t r[2 * PPW];
    // a barrier that orders this wave's LDS accesses around it but, unlike
    // __syncthreads(), does not wait for the loads still landing in LDS
    auto barrier = []() { asm volatile("s_barrier" ::: "memory"); };
    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    using I2 = std::integral_constant<int, 2>;
    using I3 = std::integral_constant<int, 3>;
    // Every step issues one stage of loads (stages past the last one read
    // out of range: no memory traffic, zeros into a slot nobody reads), so
    // the count of loads younger than a given stage is the same at every
    // step and the wait before each barrier is a fixed vmcnt.
    auto prologue = [&](auto I) {
        constexpr int st = decltype(I)::value;
        if constexpr (st < D) {
            stage_idx(st, r);
            dma(I, st, r);
        }
    };
    prologue(I0{});
    prologue(I1{});
    prologue(I2{});
    prologue(I3{});
    stage_idx(D, r);
    wait_vmcnt_le<(D - 1) * PER_STAGE>();
    barrier();
    // stage t lives in slot t % S; the loop is unrolled by S so that every
    // slot is a compile-time choice of LDS object
    auto step = [&](auto I, int t) {
        constexpr int slot = decltype(I)::value;
        // refill the slot consumed in the previous stage (freed by the barrier)
        dma(std::integral_constant<int, (slot + D) % S>{}, t + D, r);
        stage_idx(t + D + 1, r);
        const char *la = stage_a(I), *lb = stage_b(I);
#pragma unroll
        for (int ks = 0; ks < BKS / 16; ++ks) {
            bf16x8_t a[FM], b[FN];
            using RA = std::integral_constant<int, ROWB>;
            using RBB = std::integral_constant<int, ROWBB>;
#pragma unroll
            for (int i = 0; i < FM; ++i) a[i] = frag(la + aoff[i] + ks * 16 * ROWB, RA{});
#pragma unroll
            for (int j = 0; j < FN; ++j) b[j] = frag(lb + boff[j] + ks * 16 * ROWBB, RBB{});
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int i = 0; i < FM; ++i)
                    acc[j][i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[j], a[i], acc[j][i], 0, 0, 0);
        }
        // stage t+1 must have landed for every wave before the barrier;
        // stages t+2 .. t+D may stay in flight
        wait_vmcnt_le<(D - 1) * PER_STAGE>();
        barrier();
    };
    int t0 = 0;
    for (; t0 + S <= nT; t0 += S) {
        step(I0{}, t0);
        step(I1{}, t0 + 1);
        if constexpr (S > 2) step(I2{}, t0 + 2);
        if constexpr (S > 3) step(I3{}, t0 + 3);
    }
    if (t0 < nT) step(I0{}, t0);
    if (t0 + 1 < nT) step(I1{}, t0 + 1);
    if constexpr (S > 2) { if (t0 + 2 < nT) step(I2{}, t0 + 2); }
    wait_vmcnt_le<0>();   // the out-of-range tail loads, before the block can exit

    // acc[j][i][4*gq + r]: n = n0 + wn*TWN + 32j + 8gq + 4*(lane/32) + r,
    //                      m = m0 + wm*128 + 32i + lane%32
    const int lr = lane & 31, lh = lane >> 5;
    if constexpr (EPI == 1) {
        static_assert(NW == 8 && FM == 4 && FN == 2 && BT == 256 && BNT == 256 && BKS >= 32,
                      "SwiGLU epilogue layout");
        typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
        typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
        auto obj = [&](int q) -> char * {
            return q == 0 ? sA0 : q == 1 ? sA1 : q == 2 ? sB0 : sB1;
        };
        const int F = N / 2, c0 = n0 / 2;
        // thread role: channel pair cp (channels c0 + 2cp, +1), row group g8
        // (rows 8*g8 .. +7 and 64 + 8*g8 .. +7 of a pass's 128)
        const int cp = tid >> 3, g8 = tid & 7;
        double eA = 0.0, eB = 0.0;
        uint32_t hk[2][2][2][4];                 // [pass][half][channel][8 packed rows]
        __syncthreads();                         // ring reads done, tail loads landed
#pragma unroll
        for (int p = 0; p < 2; ++p) {
            // pass p: rows m0 + 128p .. +127 (the waves with wm == p), object i
            // holding rows 32i .. 32i+31 of the pass; within a row the 16-byte
            // chunk c sits at c ^ (row % 32)
            if (wm == p) {
#pragma unroll
                for (int i = 0; i < FM; ++i)
#pragma unroll
                    for (int j = 0; j < FN; ++j)
#pragma unroll
                        for (int gq = 0; gq < 4; ++gq) {
                            const int c = (wn * TWN) / 8 + 4 * j + gq;
                            const u32x2_t v = {pack_bf16x2(acc[j][i][4 * gq], acc[j][i][4 * gq + 1]),
                                               pack_bf16x2(acc[j][i][4 * gq + 2], acc[j][i][4 * gq + 3])};
                            *reinterpret_cast<u32x2_t *>(obj(i) + lr * ROWB + 16 * (c ^ lr) + 8 * lh) = v;
                        }
            }
            __syncthreads();
            const int mp = m0 + 128 * p;
#pragma unroll
            for (int half = 0; half < 2; ++half) {
                const int R0 = 64 * half + 8 * g8;          // first of the thread's 8 rows
                const char *o = obj(R0 / 32);
                uint32_t *hA = hk[p][half][0], *hB = hk[p][half][1];
#pragma unroll
                for (int r = 0; r < 8; ++r) {
                    const int rl = (R0 % 32) + r;           // row within the object
                    const uint32_t gw = *reinterpret_cast<const uint32_t *>(
                        o + rl * ROWB + 16 * ((cp >> 2) ^ rl) + 4 * (cp & 3));
                    const uint32_t uw = *reinterpret_cast<const uint32_t *>(
                        o + rl * ROWB + 16 * ((16 + (cp >> 2)) ^ rl) + 4 * (cp & 3));
                    const uint32_t a = swiglu_bf16(gw & 0xffffu, uw & 0xffffu);
                    const uint32_t b = swiglu_bf16(gw >> 16, uw >> 16);
                    if (r & 1) { hA[r >> 1] |= a << 16; hB[r >> 1] |= b << 16; }
                    else { hA[r >> 1] = a; hB[r >> 1] = b; }
                }
                // M % 8 == 0: the 8 rows are all inside or all past M
                if (mp + R0 < M) {
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const double a0 = static_cast<double>(__uint_as_float(hA[q] << 16));
                        const double a1 = static_cast<double>(__uint_as_float(hA[q] & 0xffff0000u));
                        const double b0 = static_cast<double>(__uint_as_float(hB[q] << 16));
                        const double b1 = static_cast<double>(__uint_as_float(hB[q] & 0xffff0000u));
                        eA = fma(a0, a0, eA); eA = fma(a1, a1, eA);
                        eB = fma(b0, b0, eB); eB = fma(b1, b1, eB);
                    }
                }
            }
            __syncthreads();                     // the staged rows are read
        }
        // H^T of the tile through the same objects: channel row c (0..127) in
        // object c / 32, row c % 32; its 16-byte chunk q (8 tokens) at q ^ (c % 32)
#pragma unroll
        for (int p = 0; p < 2; ++p)
#pragma unroll
            for (int half = 0; half < 2; ++half)
#pragma unroll
                for (int ch = 0; ch < 2; ++ch) {
                    const int c = 2 * cp + ch, q = 16 * p + 8 * half + g8;
                    const uint32_t *h = hk[p][half][ch];
                    *reinterpret_cast<u32x4_t *>(obj(c >> 5) + (c & 31) * ROWB + 16 * (q ^ (c & 31))) =
                        u32x4_t{h[0], h[1], h[2], h[3]};
                }
        __syncthreads();
        {
            // each half-wave writes one channel row per pass: 32 lanes x 16
            // bytes = the tile's 256 tokens (streaming stores, as Y's)
            uint16_t *Hu = Y + unit * static_cast<int64_t>(F) * ldy + m0;
            const int q = lane & 31, hw = tid >> 5;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int c = hw + 16 * i;
                const u32x4_t v = *reinterpret_cast<const u32x4_t *>(obj(c >> 5) + (c & 31) * ROWB +
                                                                     16 * (q ^ (c & 31)));
                if (m0 + 8 * q < M)
                    __builtin_nontemporal_store(v, reinterpret_cast<u32x4_t *>(
                        Hu + static_cast<int64_t>(c0 + c) * ldy + 8 * q));
            }
        }
        // the 8 row groups of a channel pair are lanes 8q .. 8q+7: add them
        // (lane ^ 1, lane ^ 2, then the mirror within 8 lanes; every lane of
        // the group ends with the same sum)
        eA += dpp_f64<0xB1>(eA);  eB += dpp_f64<0xB1>(eB);
        eA += dpp_f64<0x4E>(eA);  eB += dpp_f64<0x4E>(eB);
        eA += dpp_f64<0x141>(eA); eB += dpp_f64<0x141>(eB);
        if (g8 == 0) {
            double *pp = part + (unit * tiles_m + m0 / BT) * static_cast<int64_t>(F) + c0 + 2 * cp;
            pp[0] = eA;
            pp[1] = eB;
        }
        return;
    }
    uint16_t *Yu = Y + unit * static_cast<int64_t>(M) * ldy;
    const int rows = min(BT, M - m0);
    const __amdgpu_buffer_rsrc_t yr = __builtin_amdgcn_make_buffer_rsrc(
        Yu + static_cast<int64_t>(m0) * ldy, 0, static_cast<uint32_t>(rows * ldy * 2), 0x00020000);
    if (BNT == 256 && vec_y == 2 && n0 + BT <= N) {
        // Whole-width tile with 16-byte aligned rows: the tile goes out in two
        // passes through the (now idle) ring, so that every store writes 16
        // bytes of a 512-byte row run.  Pass p holds fragments i = 2p, 2p+1 of
        // every wave: 128 rows, 32 per ring object; within a row the 16-byte
        // chunk c sits at position c ^ (row % 32).
        static_assert(FM == 4 && BT == 256 && (BNT == 256 || BNT == 128), "staged epilogue layout");
        auto obj = [&](int q) -> char * {
            return q == 0 ? sA0 : q == 1 ? sA1 : q == 2 ? sB0 : sB1;
        };
        __syncthreads();                      // ring reads done, tail loads landed
#pragma unroll
        for (int p = 0; p < 2; ++p) {
#pragma unroll
            for (int ii = 0; ii < 2; ++ii) {
                const int i = 2 * p + ii;
                char *o = obj(2 * wm + ii);
#pragma unroll
                for (int j = 0; j < FN; ++j)
#pragma unroll
                    for (int gq = 0; gq < 4; ++gq) {
                        const int c = (wn * TWN) / 8 + 4 * j + gq;
                        typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
                        const u32x2_t v = {pack_bf16x2(acc[j][i][4 * gq], acc[j][i][4 * gq + 1]),
                                           pack_bf16x2(acc[j][i][4 * gq + 2], acc[j][i][4 * gq + 3])};
                        *reinterpret_cast<u32x2_t *>(o + lr * ROWB + 16 * (c ^ lr) + 8 * lh) = v;
                    }
            }
            __syncthreads();
            // wave w stores half-tile rows 16w .. 16w+15, two rows per instruction
            const char *o = obj(wave / 2);
            const int c = lane & 31;
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const int rl = 16 * (wave & 1) + 2 * q + lh;          // row within the object
                const int R = 16 * wave + 2 * q + lh;                 // row within the half tile
                const int ml = (R / 64) * 128 + 64 * p + (R % 64);
                typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
                const u32x4_t v = *reinterpret_cast<const u32x4_t *>(o + rl * ROWB + 16 * (c ^ rl));
                // streaming (nt) stores: Y is not read again here, and keeping it
                // out of L2 leaves the operand panels there (measured 2 % faster)
                __builtin_amdgcn_raw_buffer_store_b128(v, yr, static_cast<uint32_t>((ml * ldy + n0 + 8 * c) * 2), 0, 2);
            }
            if (p == 0) __syncthreads();      // pass 1 overwrites the staged rows
        }
        return;
    }
    const bool full_n = vec_y && n0 + BNT <= N;
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int i = 0; i < FM; ++i) {
            const int ml = wm * 128 + 32 * i + lr;      // rows past M fall outside yr
#pragma unroll
            for (int gq = 0; gq < 4; ++gq) {
                const int n = n0 + wn * TWN + 32 * j + 8 * gq + 4 * lh;
                const uint32_t w0 = pack_bf16x2(acc[j][i][4 * gq], acc[j][i][4 * gq + 1]);
                const uint32_t w1 = pack_bf16x2(acc[j][i][4 * gq + 2], acc[j][i][4 * gq + 3]);
                const uint32_t off = static_cast<uint32_t>((ml * ldy + n) * 2);
                if (full_n) {
                    typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
                    __builtin_amdgcn_raw_buffer_store_b64(u32x2_t{w0, w1}, yr, off, 0, 0);
                } else {
                    const uint16_t e[4] = {static_cast<uint16_t>(w0), static_cast<uint16_t>(w0 >> 16),
                                           static_cast<uint16_t>(w1), static_cast<uint16_t>(w1 >> 16)};
#pragma unroll
                    for (int rr = 0; rr < 4; ++rr)
                        if (n + rr < N)
                            __builtin_amdgcn_raw_buffer_store_b16(e[rr], yr, off + 2 * rr, 0, 0);
                }
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

constexpr int kBigWaves = 4;

hipError_t launch_gemm_bf16(const uint16_t *X, const uint16_t *W, const int32_t *idx,
                            int64_t B, int64_t M, int64_t N, int64_t K, int64_t k,
                            int64_t ldx, int64_t ldw, uint16_t *Y, int64_t ldy,
                            hipStream_t stream) {
    (void)K;
    const bool vec = (reinterpret_cast<uintptr_t>(W) % 16 == 0) && (ldw % 8 == 0);
    const int64_t big_tiles = ((M + big::BM - 1) / big::BM) * ((N + big::BN - 1) / big::BN);
    const int64_t w_bytes = K * ldw * 2;
    const bool offsets_fit = static_cast<int64_t>(big::BM + 1) * ldx * 2 < (int64_t(1) << 31) &&
                             w_bytes + ldw * 2 < (int64_t(1) << 31);
    if (vec && offsets_fit && big_tiles * B >= 128) {
        const int tm = static_cast<int>((M + big::BM - 1) / big::BM);
        const int tn = static_cast<int>((N + big::BN - 1) / big::BN);
        dim3 grid(static_cast<unsigned>(tm * tn), static_cast<unsigned>(B));
        hipLaunchKernelGGL(gemm_gather_bf16_big_kernel<kBigWaves>, grid, dim3(kBigWaves * 64), 0,
                           stream, X, W, idx, Y, static_cast<int>(M), static_cast<int>(N),
                           static_cast<int>(k), ldx, ldw, ldy, w_bytes, tm, tn);
        return hipGetLastError();
    }
    constexpr int BM = 128, BN = 128, BK = 32, WM = 2, WN = 2;
    dim3 grid(static_cast<unsigned>((N + BN - 1) / BN), static_cast<unsigned>((M + BM - 1) / BM),
              static_cast<unsigned>(B));
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

constexpr int kKmajorWaves = 8;
constexpr int kTrWaves = 8, kTrRows = 32, kTrStages = 3;

namespace {

// The K-major GEMM over B units; units u read W + (u / w_ugroup) * w_ustride.
// Grouped weights and K-loop trimming exist only in the large-tile kernel,
// which then serves small problems too; hipErrorNotSupported (nothing
// launched) when they are asked for with Y rows too long for its addressing.
hipError_t kmajor_dispatch(const uint16_t *Xt, const uint16_t *W, const int32_t *idx, int64_t B,
                           int64_t M, int64_t N, int64_t K, int64_t k, int64_t ldxt, int64_t ldw,
                           uint16_t *Y, int64_t ldy, int64_t w_ustride, int w_ugroup,
                           int trim, int64_t trim_off, hipStream_t stream) {
    const int64_t xt_bytes = K * ldxt * 2, w_bytes = K * ldw * 2;
    const int64_t t256 = ((M + 255) / 256) * ((N + 255) / 256);
    const bool grouped = (w_ustride != 0 && w_ugroup < B) || trim;
    // Y rows of one 256-row tile are addressed with 32-bit byte offsets
    if ((t256 * B >= 128 || grouped) && ldy < (int64_t(1) << 23)) {
        const int vec_y = (reinterpret_cast<uintptr_t>(Y) % 16 == 0 && ldy % 8 == 0) ? 2
                          : (reinterpret_cast<uintptr_t>(Y) % 8 == 0 && ldy % 4 == 0) ? 1 : 0;
        const int tm = static_cast<int>((M + 255) / 256);
        if (N <= 128) {
            // 256 x 128 tiles: no half-empty tile, two workgroups per CU
            hipLaunchKernelGGL((gemm_kmajor_tr_kernel<4, kTrRows, kTrStages, 0, 128, 2>),
                               dim3(tm, static_cast<unsigned>(B)), dim3(4 * 64), 0, stream,
                               Xt, W, idx, Y, static_cast<int>(M), static_cast<int>(N),
                               static_cast<int>(k), ldxt, ldw, ldy, xt_bytes, w_bytes, tm, 1, vec_y,
                               nullptr, w_ustride, w_ugroup, trim, trim_off);
            return hipGetLastError();
        }
        const int tn = static_cast<int>((N + 255) / 256);
        hipLaunchKernelGGL((gemm_kmajor_tr_kernel<kTrWaves, kTrRows, kTrStages>),
                           dim3(tm * tn, static_cast<unsigned>(B)), dim3(kTrWaves * 64), 0, stream,
                           Xt, W, idx, Y, static_cast<int>(M), static_cast<int>(N),
                           static_cast<int>(k), ldxt, ldw, ldy, xt_bytes, w_bytes, tm, tn, vec_y,
                           nullptr, w_ustride, w_ugroup, trim, trim_off);
        return hipGetLastError();
    }
    if (grouped) return hipErrorNotSupported;
    if (t256 * B >= 128) {
        const int tm = static_cast<int>((M + 255) / 256), tn = static_cast<int>((N + 255) / 256);
        hipLaunchKernelGGL((gemm_kmajor_bf16_kernel<256, kKmajorWaves>),
                           dim3(tm * tn, static_cast<unsigned>(B)), dim3(kKmajorWaves * 64), 0, stream, Xt, W, idx, Y, static_cast<int>(M),
                           static_cast<int>(N), static_cast<int>(K), static_cast<int>(k), ldxt,
                           ldw, ldy, xt_bytes, w_bytes, tm, tn);
    } else {
        const int tm = static_cast<int>((M + 127) / 128), tn = static_cast<int>((N + 127) / 128);
        hipLaunchKernelGGL((gemm_kmajor_bf16_kernel<128, 4>),
                           dim3(tm * tn, static_cast<unsigned>(B)), dim3(256), 0, stream, Xt, W, idx, Y, static_cast<int>(M),
                           static_cast<int>(N), static_cast<int>(K), static_cast<int>(k), ldxt,
                           ldw, ldy, xt_bytes, w_bytes, tm, tn);
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_kmajor_bf16(const uint16_t *Xt, const uint16_t *W, const int32_t *idx,
                                  int64_t B, int64_t M, int64_t N, int64_t K, int64_t k,
                                  int64_t ldxt, int64_t ldw, uint16_t *Y, int64_t ldy,
                                  hipStream_t stream) {
    return kmajor_dispatch(Xt, W, idx, B, M, N, K, k, ldxt, ldw, Y, ldy, 0, 1, 0, 0, stream);
}

hipError_t launch_gemm_kmajor_grouped_bf16(const uint16_t *Xt, const uint16_t *W, const int32_t *idx,
                                          int64_t B, int64_t M, int64_t N, int64_t K, int64_t k,
                                          int64_t ldxt, int64_t ldw, uint16_t *Y, int64_t ldy,
                                          int64_t w_ustride, int w_ugroup, int trim, int64_t trim_off,
                                          hipStream_t stream) {
    return kmajor_dispatch(Xt, W, idx, B, M, N, K, k, ldxt, ldw, Y, ldy, w_ustride, w_ugroup, trim,
                           trim_off, stream);
}

hipError_t launch_gemm_swiglu_kmajor_bf16(const uint16_t *Xt, const uint16_t *W,
                                         const int32_t *idx, int64_t B, int64_t M, int64_t F,
                                         int64_t K, int64_t k, int64_t ldxt, int64_t ldw,
                                         uint16_t *Ht, int64_t ldht, double *energy,
                                         double *partials, hipStream_t stream) {
    const int64_t xt_bytes = K * ldxt * 2, w_bytes = K * ldw * 2;
    const int tm = static_cast<int>((M + 255) / 256), tn = static_cast<int>(F / 128);
    hipLaunchKernelGGL((gemm_kmajor_tr_kernel<kTrWaves, kTrRows, kTrStages, 1>),
                       dim3(tm * tn, static_cast<unsigned>(B)), dim3(kTrWaves * 64), 0, stream,
                       Xt, W, idx, Ht, static_cast<int>(M), static_cast<int>(2 * F),
                       static_cast<int>(k), ldxt, ldw, ldht, xt_bytes, w_bytes, tm, tn, 2, partials);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // energies: the row tiles' partial sums, added in tile order
    return launch_score_finalize(partials, B, tm, F, energy, stream);
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
