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

// ------------------------------------------------------- row-streaming kernel
// One workgroup per (head, 128-query tile) walks the key tiles (BT keys:
// 128 with 4 waves, or 256 with 8 waves) of its rows.
// Q and K rows (D values, 16-byte chunks) are read whole and staged in LDS
// with an odd row stride of D/2+1 words, so 32 rows read at one column hit
// 32 distinct banks; the MFMA operands are gathered from the staged rows at
// the retained dims (a zeroed pad word stands in for padding positions).
// Q's fragments are gathered once and kept in registers.  The waves split
// the 128 x BT tile into KW key strips and WQ query strips: with few retained
// dims (KSMAX k-steps) one strip of 32 keys per wave against all 128
// queries, so no K fragment is gathered twice; with more, two query strips
// keep Q's register footprint in bounds.  The product is
// formed transposed (keys x queries), so each lane holds 4 consecutive keys
// of one query; tiles are staged through LDS and written as coalesced
// 16-byte stores, BT*2-byte row pieces (the longer pieces of the 256-key
// tiles write faster).  Key tiles wholly above the diagonal are streamed
// as -inf.
namespace rowk {
constexpr int BQ = 128;       // queries per block
// cache policy of the score stores (sc1).  Streaming (nt) stores measured
// about 25% slower for this pattern of 256-byte row pieces 2*Lk bytes apart.
constexpr int kStoreAux = 16;
}  // namespace rowk

// ST: also write each score row's softmax statistics over the stored bf16
// scores of its kept keys: rmax[row] = their maximum, rinv[row] = 1 / sum of
// exp(s - rmax) (0 and 0 for a row with nothing kept).  They are taken where
// the staged tile is read back for its stores: each thread keeps, for each of
// its rows, a running maximum over its 8-key chunks and a sum rescaled when
// the maximum rises; a row's threads are consecutive lanes, merged at the end
// in a fixed butterfly.
template <int D, int KSMAX, int WQ, int NTT, int BTT, bool ST = false>
__global__ __launch_bounds__(NTT, NTT == 256 ? 2 : 1) void qk_bf16_rows_kernel(
    const uint16_t *__restrict__ Q, const uint16_t *__restrict__ Kc,
    const int32_t *__restrict__ idx, uint16_t *__restrict__ S, int H, int Hkv, int Lq, int Lk,
    int k, float scale, int causal, float *__restrict__ rmax = nullptr,
    float *__restrict__ rinv = nullptr) {
    constexpr int BQ = rowk::BQ, BT = BTT, NT = NTT;
    constexpr int OS = BT + 8;             // staged output row (16-byte aligned)
    typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
    constexpr int kStoreAux = rowk::kStoreAux;
    constexpr int RW = D / 2 + 1;          // words per staged row (odd)
    constexpr int CH = D / 8;              // 16-byte chunks per row
    constexpr int PER_T = BT * CH / NT;    // chunks staged per thread
    constexpr int KW = NT / 64 / WQ;       // waves along keys
    constexpr int FI = BT / KW / 32;       // 32-key fragments per wave
    constexpr int FJ = BQ / WQ / 32;       // 32-query fragments per wave
    static_assert(D % 16 == 0 && BT % BQ == 0 && (BT * CH) % NT == 0, "shape");
    static_assert(KSMAX * 16 <= D && (WQ == 1 || WQ == 2), "shape");

    __shared__ uint32_t rows_lds[BT * RW];
    __shared__ __attribute__((aligned(16))) uint16_t out_lds[BQ * OS];
    __shared__ __attribute__((aligned(16))) uint16_t col_off[D + 16];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int bh = blockIdx.y, b = bh / H, h = bh % H, g = h / (H / Hkv);
    // causal: the last query tiles carry the most key tiles, so they are
    // dealt first (longest work first keeps the tail of the grid short)
    const int qt = causal ? static_cast<int>(gridDim.x) - 1 - static_cast<int>(blockIdx.x) : blockIdx.x;
    const int q0 = qt * BQ;
    const int off = Lk - Lq;
    const int32_t *I = idx + static_cast<int64_t>(bh) * k;
    uint16_t *Sh = S + static_cast<int64_t>(bh) * Lq * Lk;
    const int n_tiles = (Lk + BT - 1) / BT;
    int n_compute = n_tiles;
    if (causal) {
        const int limit = min(q0 + BQ, Lq) - 1 + off;   // largest key any row keeps
        n_compute = limit < 0 ? 0 : min(n_tiles, limit / BT + 1);
    }
    constexpr int CPR = BT / 8, RPP = NT / CPR;        // 16-byte chunks per row piece, rows per pass
    const int r16 = tid / CPR, c16 = tid % CPR;         // store role: rows r16 + RPP*i, chunk c16
    // the block's rows of S; rows at or past Lq fall outside the range and are dropped
    const __amdgpu_buffer_rsrc_t sr = __builtin_amdgcn_make_buffer_rsrc(
        Sh + static_cast<int64_t>(q0) * Lk, 0, static_cast<uint32_t>(min(BQ, Lq - q0) * Lk * 2),
        0x00020000);
    constexpr int SR = BQ / RPP;              // rows per thread in the store role
    float st_m[SR], st_l[SR];                 // their running statistics (ST)
#pragma unroll
    for (int i = 0; i < SR; ++i) { st_m[i] = -__builtin_inff(); st_l[i] = 0.f; }

    if (n_compute > 0) {
        const int kp = (k + 15) & ~15;
        const int KS = kp / 16;
        for (int t = tid; t < D + 16; t += NT) col_off[t] = static_cast<uint16_t>((t < k ? I[t] : D) * 2);
        for (int r = tid; r < BT; r += NT) rows_lds[r * RW + D / 2] = 0u;

        const __amdgpu_buffer_rsrc_t qr = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint16_t *>(Q + (static_cast<int64_t>(bh) * Lq + q0) * D), 0,
            static_cast<uint32_t>(min(BQ, Lq - q0) * D * 2), 0x00020000);
        const uint16_t *Kh = Kc + (static_cast<int64_t>(b) * Hkv + g) * Lk * D;

        uint4 regs[PER_T];
        auto load_rows = [&](__amdgpu_buffer_rsrc_t rs) {
#pragma unroll
            for (int i = 0; i < PER_T; ++i) {
                const int v = tid + NT * i;
                const auto x = __builtin_amdgcn_raw_buffer_load_b128(
                    rs, static_cast<uint32_t>(((v / CH) * D + (v % CH) * 8) * 2), 0, 0);
                regs[i] = make_uint4(x[0], x[1], x[2], x[3]);
            }
        };
        auto store_rows = [&]() {
#pragma unroll
            for (int i = 0; i < PER_T; ++i) {
                const int v = tid + NT * i;
                uint32_t *dst = rows_lds + (v / CH) * RW + (v % CH) * 4;
                dst[0] = regs[i].x; dst[1] = regs[i].y; dst[2] = regs[i].z; dst[3] = regs[i].w;
            }
        };
        auto key_rsrc = [&](int kt) {
            const int t0 = kt * BT;
            return __builtin_amdgcn_make_buffer_rsrc(
                const_cast<uint16_t *>(Kh + static_cast<int64_t>(t0) * D), 0,
                static_cast<uint32_t>(min(BT, Lk - t0) * D * 2), 0x00020000);
        };
        // 8 retained dims (k-step ks, lane half) of staged row `row`
        auto frag = [&](int row, int ks) -> bf16x8_t {
            const uint4 co = *reinterpret_cast<const uint4 *>(&col_off[ks * 16 + 8 * (lane >> 5)]);
            const char *base = reinterpret_cast<const char *>(rows_lds + row * RW);
            const uint32_t o[4] = {co.x, co.y, co.z, co.w};
            uint32_t w[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint32_t lo = *reinterpret_cast<const uint16_t *>(base + (o[q] & 0xffffu));
                const uint32_t hi = *reinterpret_cast<const uint16_t *>(base + (o[q] >> 16));
                w[q] = lo | (hi << 16);
            }
            return __builtin_bit_cast(bf16x8_t, make_uint4(w[0], w[1], w[2], w[3]));
        };

        const int wk = wave / WQ, wq = wave % WQ;   // wave: BT/KW keys x BQ/WQ queries
        const int lr = lane & 31, lh = lane >> 5;

        load_rows(qr);
        store_rows();
        __syncthreads();
        bf16x8_t qf[FJ][KSMAX];
#pragma unroll
        for (int j = 0; j < FJ; ++j)
#pragma unroll
            for (int ks = 0; ks < KSMAX; ++ks)
                if (ks < KS) qf[j][ks] = frag((wq * FJ + j) * 32 + lr, ks);
        // Each block walks its key tiles starting at a tile of its own and
        // wrapping around, so that at any moment the blocks store to
        // different column ranges of their rows (all starting at column 0
        // measured about 1.5x slower without the causal mask: the row pieces
        // of simultaneous tiles then share too few memory channels).
        const int rot = (bh * 5 + qt) % n_compute;
        auto tile_at = [&](int i) { const int t = i + rot; return t >= n_compute ? t - n_compute : t; };
        load_rows(key_rsrc(tile_at(0)));
        __syncthreads();
        store_rows();
        __syncthreads();

        for (int it = 0; it < n_compute; ++it) {
            const int kt = tile_at(it);
            if (it + 1 < n_compute) load_rows(key_rsrc(tile_at(it + 1)));
            f32x16_t acc[FI][FJ];
#pragma unroll
            for (int i = 0; i < FI; ++i)
#pragma unroll
                for (int j = 0; j < FJ; ++j)
#pragma unroll
                    for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;
#pragma unroll
            for (int ks = 0; ks < KSMAX; ++ks) {
                if (ks < KS) {
#pragma unroll
                    for (int i = 0; i < FI; ++i) {
                        const bf16x8_t kf = frag((wk * FI + i) * 32 + lr, ks);
#pragma unroll
                        for (int j = 0; j < FJ; ++j)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[j][ks], acc[i][j], 0, 0, 0);
                    }
                }
            }
            // acc[i][j][4*gq + r]: key (wk*FI + i)*32 + 8*gq + 4*lh + r, query (wq*FJ + j)*32 + lr
            // a tile whose last key is at most its first query + off has no masked entry
            const bool tile_open = !causal || kt * BT + BT - 1 <= q0 + off;
#pragma unroll
            for (int i = 0; i < FI; ++i)
#pragma unroll
                for (int j = 0; j < FJ; ++j) {
                    const int ql = (wq * FJ + j) * 32 + lr;
                    const int qg = q0 + ql;
#pragma unroll
                    for (int gq = 0; gq < 4; ++gq) {
                        const int kl = (wk * FI + i) * 32 + 8 * gq + 4 * lh;
                        uint32_t w0 = pack_bf16x2(acc[i][j][4 * gq] * scale, acc[i][j][4 * gq + 1] * scale);
                        uint32_t w1 = pack_bf16x2(acc[i][j][4 * gq + 2] * scale, acc[i][j][4 * gq + 3] * scale);
                        if (!tile_open) {
                            const int lim = qg + off - (kt * BT + kl);   // keys kl + r kept iff r <= lim
                            if (lim < 0) w0 = (w0 & 0xffff0000u) | kBf16NegInf;
                            if (lim < 1) w0 = (w0 & 0x0000ffffu) | (static_cast<uint32_t>(kBf16NegInf) << 16);
                            if (lim < 2) w1 = (w1 & 0xffff0000u) | kBf16NegInf;
                            if (lim < 3) w1 = (w1 & 0x0000ffffu) | (static_cast<uint32_t>(kBf16NegInf) << 16);
                        }
                        *reinterpret_cast<uint2 *>(&out_lds[ql * OS + kl]) = make_uint2(w0, w1);
                    }
                }
            lds_barrier();
            const int col = kt * BT + c16 * 8;
            uint4 staged[BQ / RPP];
#pragma unroll
            for (int i = 0; i < BQ / RPP; ++i) {
                const int r = r16 + RPP * i;
                // unconditional (a column past Lk goes out of range): a branch
                // here would make the compiler's wait for the next K rows also
                // wait for these stores
                const uint32_t off = col < Lk ? static_cast<uint32_t>((r * Lk + col) * 2) : 0x80000000u;
                const uint4 v = *reinterpret_cast<const uint4 *>(&out_lds[r * OS + c16 * 8]);
                __builtin_amdgcn_raw_buffer_store_b128(u32x4_t{v.x, v.y, v.z, v.w}, sr, off, 0, kStoreAux);
                staged[i] = v;
            }
            if constexpr (ST) {
                // After the stores are issued, so that this work overlaps their
                // drain, and without branches, for the same reason as above.
                // Masked keys hold -inf already; a chunk past Lk is not scores.
#pragma unroll
                for (int i = 0; i < BQ / RPP; ++i) {
                    const uint32_t w[4] = {staged[i].x, staged[i].y, staged[i].z, staged[i].w};
                    float e[8];
                    float cm = -__builtin_inff();
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        e[2 * q] = col < Lk ? __uint_as_float(w[q] << 16) : -__builtin_inff();
                        e[2 * q + 1] = col < Lk ? __uint_as_float(w[q] & 0xffff0000u) : -__builtin_inff();
                        cm = fmaxf(cm, fmaxf(e[2 * q], e[2 * q + 1]));
                    }
                    const float mm = fmaxf(st_m[i], cm);
                    // with nothing kept so far every term below is exp(-inf) = 0
                    const float mref = mm == -__builtin_inff() ? 0.f : mm;
                    float l = st_l[i] * __expf(st_m[i] - mref);
#pragma unroll
                    for (int q = 0; q < 8; ++q) l += __expf(e[q] - mref);
                    st_m[i] = mm;
                    st_l[i] = l;
                }
            }
            if (it + 1 < n_compute) store_rows();
            lds_barrier();
        }
    }
    if constexpr (ST) {
#pragma unroll
        for (int i = 0; i < SR; ++i) {
#pragma unroll
            for (int sh = 1; sh < CPR; sh <<= 1) {
                const float m2 = __shfl_xor(st_m[i], sh), l2 = __shfl_xor(st_l[i], sh);
                const float mm = fmaxf(st_m[i], m2);
                if (mm != -__builtin_inff()) {
                    const float a = st_m[i] == -__builtin_inff() ? 0.f : st_l[i] * __expf(st_m[i] - mm);
                    const float c = m2 == -__builtin_inff() ? 0.f : l2 * __expf(m2 - mm);
                    st_m[i] = mm;
                    st_l[i] = a + c;
                }
            }
            const int r = r16 + RPP * i;
            if (c16 == 0 && q0 + r < Lq) {
                const int64_t row = static_cast<int64_t>(bh) * Lq + q0 + r;
                const bool empty = !(st_l[i] > 0.f);
                rmax[row] = empty ? 0.f : st_m[i];
                rinv[row] = empty ? 0.f : 1.0f / st_l[i];
            }
        }
    }
    // key tiles wholly above the diagonal: one contiguous run per row, each
    // wave writing whole rows with 1 KiB per store instruction
    const uint32_t ninf2 = 0xff80ff80u;
    const int c0 = n_compute * BT;
    const int nv = (Lk - c0) / 8;                 // 16-byte vectors per row (Lk % 8 == 0)
    for (int r = wave; r < BQ; r += NT / 64)
        for (int v = lane; v < nv; v += 64)
            __builtin_amdgcn_raw_buffer_store_b128(u32x4_t{ninf2, ninf2, ninf2, ninf2}, sr,
                static_cast<uint32_t>((r * Lk + c0 + 8 * v) * 2), 0, kStoreAux);
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

bool qk_rows_ok(int64_t Lk, int64_t D, const void *S) {
    // Lk bound: a block's 128 rows of S are addressed with 32-bit byte offsets
    return (D == 64 || D == 128) && Lk % 8 == 0 && Lk <= (1 << 22) &&
           reinterpret_cast<uintptr_t>(S) % 16 == 0;
}

hipError_t launch_qk_rowstats_bf16(const uint16_t *Q, const uint16_t *Kc, const int32_t *idx,
                                   int64_t batch, int64_t H, int64_t Hkv, int64_t Lq, int64_t Lk,
                                   int64_t D, int64_t k, float scale, bool causal, uint16_t *S,
                                   float *rmax, float *rinv, hipStream_t stream) {
    if (!qk_rows_ok(Lk, D, S)) return hipErrorNotSupported;
    dim3 grid(static_cast<unsigned>((Lq + rowk::BQ - 1) / rowk::BQ), static_cast<unsigned>(batch * H));
    const bool wide = D == 128 && k <= 96;
    auto kern = D == 64 ? qk_bf16_rows_kernel<64, 4, 1, 256, 128, true>
              : k <= 64 ? qk_bf16_rows_kernel<128, 4, 1, 512, 256, true>
              : k <= 96 ? qk_bf16_rows_kernel<128, 8, 2, 512, 256, true>
                        : qk_bf16_rows_kernel<128, 8, 2, 256, 128, true>;
    hipLaunchKernelGGL(kern, grid, dim3(wide ? 512 : 256), 0, stream, Q, Kc, idx, S,
                       static_cast<int>(H), static_cast<int>(Hkv), static_cast<int>(Lq),
                       static_cast<int>(Lk), static_cast<int>(k), scale, causal ? 1 : 0, rmax, rinv);
    return hipGetLastError();
}

hipError_t launch_qk_bf16(const uint16_t *Q, const uint16_t *Kc, const int32_t *idx,
                          int64_t batch, int64_t H, int64_t Hkv, int64_t Lq, int64_t Lk,
                          int64_t D, int64_t k, float scale, bool causal, uint16_t *S,
                          hipStream_t stream) {
    const bool rows_ok = qk_rows_ok(Lk, D, S);
    if (rows_ok) {
        dim3 grid(static_cast<unsigned>((Lq + rowk::BQ - 1) / rowk::BQ),
                  static_cast<unsigned>(batch * H));
        // up to 64 retained dims: one key strip per wave; more: 2x2 strips
        // up to 96 retained dims: 256-key tiles, one 8-wave block per CU, so
        // that every stored row piece is 512 bytes; more dims: 128-key tiles,
        // two 4-wave blocks per CU (the heavier product overlaps better)
        const bool wide = D == 128 && k <= 96;
        auto kern = D == 64 ? qk_bf16_rows_kernel<64, 4, 1, 256, 128>
                  : k <= 64 ? qk_bf16_rows_kernel<128, 4, 1, 512, 256>
                  : k <= 96 ? qk_bf16_rows_kernel<128, 8, 2, 512, 256>
                            : qk_bf16_rows_kernel<128, 8, 2, 256, 128>;
        hipLaunchKernelGGL(kern, grid, dim3(wide ? 512 : 256), 0, stream, Q, Kc, idx, S,
                           static_cast<int>(H), static_cast<int>(Hkv), static_cast<int>(Lq),
                           static_cast<int>(Lk), static_cast<int>(k), scale, causal ? 1 : 0,
                           nullptr, nullptr);
        return hipGetLastError();
    }
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
