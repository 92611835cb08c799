// Reduced attention block: O = softmax(S + M) V with the reduced scores
// S[h] = scale * Q[h][:, I_h] K[g(h)][:, I_h]^T of Sec. 3.3 (GQA: query head h
// reads kv head h / (H / Hkv)), computed tile by tile with an online softmax
// so that S never reaches memory.
//
// One workgroup per (head, 128 queries); each of its four waves owns 32
// queries and walks the key tiles (64 keys) the causal mask leaves it:
//   * Q rows are staged once in LDS (odd row stride) and each wave gathers its
//     queries' retained dims into registers; K rows are staged per tile the
//     same way and gathered at the retained dims;
//   * the scores are formed transposed (keys x queries, v_mfma_f32_32x32x16_bf16),
//     so a lane holds 16 keys of one query: the row max and row sum need one
//     exchange with the partner lane 32 away, and the lane's probabilities,
//     rounded to bf16, are directly the second MFMA operand of O^T += V^T P^T;
//   * V rows are staged with their 16-byte chunks at c ^ 4*(row % 4) and
//     read with the gfx950 transposing LDS read, which yields the
//     4-consecutive-keys-per-lane layout the probabilities are in;
//   * O^T is accumulated in fp32 (a lane holds 16 output dims of one query),
//     rescaled by its own query's exp(m_old - m_new), and divided by the row
//     sum at the end.  A query with no unmasked key gets 0.
#include "device_common.h"
#include "kernels.h"

namespace rmm {

namespace {

namespace attk {
constexpr int BQ = 128, BT = 64, NT = 256, D = 128;
constexpr int RW = D / 2 + 1;              // words per staged Q/K row (odd)
constexpr int CH = D / 8;                  // 16-byte chunks per row
constexpr int VROW = D * 2;                // bytes per staged V row
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
constexpr float kLog2e = 1.4426950408889634f;
}  // namespace attk

template <int KSMAX>
__global__ __launch_bounds__(attk::NT, 2) void attn_bf16_kernel(
    const uint16_t *__restrict__ Q, const uint16_t *__restrict__ Kc,
    const uint16_t *__restrict__ V, const int32_t *__restrict__ idx, uint16_t *__restrict__ O,
    int H, int Hkv, int Lq, int Lk, int k, float scale, int causal) {
    using namespace attk;
    constexpr int KROWS_T = BT * CH / NT;      // 16-byte K (or V) chunks per thread per tile
    constexpr int QROWS_T = BQ * CH / NT;      // 16-byte Q chunks per thread
    static_assert(KSMAX * 16 <= D && KROWS_T * NT == BT * CH, "shape");

    __shared__ uint32_t rows_lds[BQ * RW];     // Q (once), then K tiles (first BT rows)
    __shared__ __attribute__((aligned(16))) char v_lds[BT * VROW];
    __shared__ __attribute__((aligned(16))) uint16_t col_off[D + 16];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int bh = blockIdx.y, b = bh / H, h = bh % H, g = h / (H / Hkv);
    // causal: the last query tiles carry the most key tiles, so they go first
    const int qt = causal ? static_cast<int>(gridDim.x) - 1 - static_cast<int>(blockIdx.x) : blockIdx.x;
    const int q0 = qt * BQ;
    const int off = Lk - Lq;
    const int32_t *I = idx + static_cast<int64_t>(bh) * k;
    const int kp = (k + 15) & ~15;
    const int KS = kp / 16;
    // key tiles any of the block's rows keeps
    int n_tiles = (Lk + BT - 1) / BT;
    if (causal) {
        const int limit = min(q0 + BQ, Lq) - 1 + off;
        n_tiles = limit < 0 ? 0 : min(n_tiles, limit / BT + 1);
    }

    for (int t = tid; t < D + 16; t += NT) col_off[t] = static_cast<uint16_t>((t < k ? I[t] : D) * 2);
    for (int r = tid; r < BQ; r += NT) rows_lds[r * RW + D / 2] = 0u;

    const __amdgpu_buffer_rsrc_t qr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t *>(Q + (static_cast<int64_t>(bh) * Lq + q0) * D), 0,
        static_cast<uint32_t>(min(BQ, Lq - q0) * D * 2), 0x00020000);
    const uint16_t *Kh = Kc + (static_cast<int64_t>(b) * Hkv + g) * Lk * D;
    const uint16_t *Vh = V + (static_cast<int64_t>(b) * Hkv + g) * Lk * D;
    // a key tile's rows as a buffer: rows past Lk read zeros (and are masked)
    auto tile_rsrc = [&](const uint16_t *base, int kt) {
        const int t0 = min(kt * BT, Lk);
        return __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint16_t *>(base + static_cast<int64_t>(t0) * D), 0,
            static_cast<uint32_t>(min(BT, Lk - t0) * D * 2), 0x00020000);
    };
    auto chunk_off = [&](int v) { return static_cast<uint32_t>(((v / CH) * D + (v % CH) * 8) * 2); };
    auto stage_rows = [&](const uint4 &x, int v) {      // Q / K row chunk -> odd-stride rows
        uint32_t *dst = rows_lds + (v / CH) * RW + (v % CH) * 4;
        dst[0] = x.x; dst[1] = x.y; dst[2] = x.z; dst[3] = x.w;
    };
    auto stage_v = [&](const uint4 &x, int v) {          // V row chunk -> swizzled chunk
        const int t = v / CH, c = v % CH;
        *reinterpret_cast<uint4 *>(v_lds + t * VROW + ((c ^ (4 * (t & 3))) * 16)) = x;
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

    const int lr = lane & 31, lh = lane >> 5;

    // Q: stage the block's rows, gather this wave's 32 queries
    {
        uint4 rq[QROWS_T];
#pragma unroll
        for (int i = 0; i < QROWS_T; ++i) {
            const auto x = __builtin_amdgcn_raw_buffer_load_b128(qr, chunk_off(tid + NT * i), 0, 0);
            rq[i] = make_uint4(x[0], x[1], x[2], x[3]);
        }
        __syncthreads();                       // col_off and the pad words are written
#pragma unroll
        for (int i = 0; i < QROWS_T; ++i) stage_rows(rq[i], tid + NT * i);
        __syncthreads();
    }
    bf16x8_t qf[KSMAX];
#pragma unroll
    for (int ks = 0; ks < KSMAX; ++ks)
        if (ks < KS) qf[ks] = frag(wave * 32 + lr, ks);

    // V^T fragment addressing (transposing read): 16-lane group gr reads rows
    // row0 + (s16 / 4) of dims 16*(gr % 2) + 4*(s16 % 4) .. +3 of a 32-dim block
    const int gr = lane >> 4, s16 = lane & 15, vv = s16 >> 2, qq = s16 & 3;
    int voff[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
        voff[db] = (4 * (gr >> 1) + vv) * VROW + ((4 * (db ^ vv) + 2 * (gr & 1) + (qq >> 1)) * 16) +
                   8 * (qq & 1);
    auto vfrag = [&](int db, int s) -> bf16x8_t {
        const char *p = v_lds + voff[db] + 16 * s * VROW;
        const s16x4_t lo = lds_read_tr16(p);
        const s16x4_t hi = lds_read_tr16(p + 8 * VROW);
        typedef short s16x8_t __attribute__((ext_vector_type(8)));
        return __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    };

    f32x16_t o_acc[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) o_acc[db][v] = 0.f;
    float m_run = -__builtin_inff(), l_run = 0.f;   // this lane's query (q = lane % 32)
    const int qg = q0 + wave * 32 + lr;
    const float sl2 = scale * kLog2e;

    uint4 rk[KROWS_T], rv[KROWS_T];
    auto load_tile = [&](int kt) {
        const __amdgpu_buffer_rsrc_t kr = tile_rsrc(Kh, kt), vr = tile_rsrc(Vh, kt);
#pragma unroll
        for (int i = 0; i < KROWS_T; ++i) {
            const auto x = __builtin_amdgcn_raw_buffer_load_b128(kr, chunk_off(tid + NT * i), 0, 0);
            rk[i] = make_uint4(x[0], x[1], x[2], x[3]);
            const auto y = __builtin_amdgcn_raw_buffer_load_b128(vr, chunk_off(tid + NT * i), 0, 0);
            rv[i] = make_uint4(y[0], y[1], y[2], y[3]);
        }
    };
    auto store_tile = [&]() {
#pragma unroll
        for (int i = 0; i < KROWS_T; ++i) {
            stage_rows(rk[i], tid + NT * i);
            stage_v(rv[i], tid + NT * i);
        }
    };
    if (n_tiles > 0) {
        load_tile(0);
        __syncthreads();                       // every wave has gathered its Q fragments
        store_tile();
        lds_barrier();
    }
    for (int kt = 0; kt < n_tiles; ++kt) {
        if (kt + 1 < n_tiles) load_tile(kt + 1);
        // S^T for the tile: s[tb][4*gq + r] = key kt*BT + 32*tb + 8*gq + 4*lh + r
        f32x16_t s[BT / 32];
#pragma unroll
        for (int tb = 0; tb < BT / 32; ++tb)
#pragma unroll
            for (int v = 0; v < 16; ++v) s[tb][v] = 0.f;
#pragma unroll
        for (int ks = 0; ks < KSMAX; ++ks) {
            if (ks < KS) {
#pragma unroll
                for (int tb = 0; tb < BT / 32; ++tb)
                    s[tb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag(32 * tb + lr, ks), qf[ks], s[tb], 0, 0, 0);
            }
        }
        // scale to log2 units and mask: key t past Lk, or (causal) past qg + off
        const int lim = causal ? min(qg + off, Lk - 1) : Lk - 1;
        float mx = -__builtin_inff();
#pragma unroll
        for (int tb = 0; tb < BT / 32; ++tb)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int t = kt * BT + 32 * tb + 8 * (v >> 2) + 4 * lh + (v & 3);
                const float x = t <= lim ? s[tb][v] * sl2 : -__builtin_inff();
                s[tb][v] = x;
                mx = fmaxf(mx, x);
            }
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float m_new = fmaxf(m_run, mx);
        const float m_use = m_new == -__builtin_inff() ? 0.f : m_new;   // nothing kept yet
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
        float lsum = 0.f;
#pragma unroll
        for (int tb = 0; tb < BT / 32; ++tb)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const float p = __builtin_amdgcn_exp2f(s[tb][v] - m_use);
                s[tb][v] = p;
                lsum += p;
            }
        lsum += __shfl_xor(lsum, 32);
        l_run = l_run * alpha + lsum;
        m_run = m_new;
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
#pragma unroll
            for (int v = 0; v < 16; ++v) o_acc[db][v] *= alpha;
        // O^T += V^T P^T over the tile's keys, 16 keys per MFMA: the lane's
        // probabilities for keys 16*st + 4*lh + {0..3} and 16*st + 8 + 4*lh + {0..3}
#pragma unroll
        for (int st = 0; st < BT / 16; ++st) {
            const int tb = st >> 1, g0 = 2 * (st & 1);
            bf16x8_t pf;
#pragma unroll
            for (int e = 0; e < 8; ++e)
                pf[e] = static_cast<__bf16>(s[tb][4 * (g0 + (e >> 2)) + (e & 3)]);
#pragma unroll
            for (int db = 0; db < D / 32; ++db)
                o_acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vfrag(db, st), pf, o_acc[db], 0, 0, 0);
        }
        lds_barrier();                         // every wave is done with this tile's K and V
        if (kt + 1 < n_tiles) store_tile();
        lds_barrier();
    }

    // O[q][d]: the lane holds d = 32*db + 8*gq + 4*lh + {0..3} of query qg
    const float inv = l_run > 0.f ? 1.f / l_run : 0.f;
    const __amdgpu_buffer_rsrc_t orr = __builtin_amdgcn_make_buffer_rsrc(
        O + (static_cast<int64_t>(bh) * Lq + q0) * D, 0,
        static_cast<uint32_t>(min(BQ, Lq - q0) * D * 2), 0x00020000);
    const int ql = wave * 32 + lr;             // rows past Lq fall outside the buffer
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int gq = 0; gq < 4; ++gq) {
            const uint32_t w0 = pack_bf16x2(o_acc[db][4 * gq] * inv, o_acc[db][4 * gq + 1] * inv);
            const uint32_t w1 = pack_bf16x2(o_acc[db][4 * gq + 2] * inv, o_acc[db][4 * gq + 3] * inv);
            __builtin_amdgcn_raw_buffer_store_b64(
                u32x2_t{w0, w1}, orr,
                static_cast<uint32_t>((ql * D + 32 * db + 8 * gq + 4 * lh) * 2), 0, 0);
        }
}

}  // namespace

hipError_t launch_attn_bf16(const uint16_t *Q, const uint16_t *Kc, const uint16_t *V,
                            const int32_t *idx, int64_t batch, int64_t H, int64_t Hkv,
                            int64_t Lq, int64_t Lk, int64_t k, float scale, bool causal,
                            uint16_t *O, hipStream_t stream) {
    dim3 grid(static_cast<unsigned>((Lq + attk::BQ - 1) / attk::BQ), static_cast<unsigned>(batch * H));
    auto kern = k <= 64 ? attn_bf16_kernel<4> : attn_bf16_kernel<8>;
    hipLaunchKernelGGL(kern, grid, dim3(attk::NT), 0, stream, Q, Kc, V, idx, O,
                       static_cast<int>(H), static_cast<int>(Hkv), static_cast<int>(Lq),
                       static_cast<int>(Lk), static_cast<int>(k), scale, causal ? 1 : 0);
    return hipGetLastError();
}

}  // namespace rmm
