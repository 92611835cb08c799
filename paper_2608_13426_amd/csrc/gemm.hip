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

hipError_t launch_gemm_kmajor_bf16(const uint16_t *Xt, const uint16_t *W, const int32_t *idx,
                                  int64_t B, int64_t M, int64_t N, int64_t K, int64_t k,
                                  int64_t ldxt, int64_t ldw, uint16_t *Y, int64_t ldy,
                                  hipStream_t stream) {
    const int64_t xt_bytes = K * ldxt * 2, w_bytes = K * ldw * 2;
    const int64_t t256 = ((M + 255) / 256) * ((N + 255) / 256);
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
