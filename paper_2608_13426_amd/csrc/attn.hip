// Reduced attention block: O = softmax(S + M) V with the reduced scores
// S[h] = scale * Q[h][:, I_h] K[g(h)][:, I_h]^T of Sec. 3.3 (GQA: query head h
// reads kv head h / (H / Hkv)); S never reaches memory.
//
// Two kernels on the caller's stream:
//   1. attn_compact_k_kernel writes, for every query head, its retained key
//      dims as contiguous rows: Ki[b][h][t][0..kp) = K[b][g(h)][t][I_h], zero
//      past k (kp = 16 * KS >= k).  This is H*Lk*kp bf16 of workspace, read
//      back once per query tile; it turns the per-tile key gather into plain
//      16-byte rows.
//   2. attn_fwd_kernel: one workgroup per (head, 256 queries), eight waves
//      of 32 queries (two per SIMD), a four-slot LDS ring of 64-key tiles
//      filled by LDS DMA two tiles ahead:
//        * S^T = Ki Q_I^T per tile (v_mfma_f32_32x32x16_bf16; Q's retained
//          dims gathered once into registers), so a lane holds 16 keys of
//          one query and the row max needs one exchange with the lane 32
//          away (v_permlane32_swap);
//        * online softmax in log2 units, exp2(fma(s, c, -m)) with
//          c = |scale| log2(e) (Q is negated exactly when scale < 0); the
//          causal mask is applied only on tiles that cross a row's limit;
//          the running max is raised (and O^T, l rescaled) only when a
//          tile's max exceeds it by more than 8 (log2 units), so weights
//          stay <= 256 and most tiles skip the rescale;
//        * O^T += V^T P^T with the weights rounded to bf16 as the MFMA's
//          second operand and V^T read with the gfx950 transposing LDS read;
//        * the two waves of a SIMD take the softmax at opposite ends of a
//          step, so one's exponentials meet the other's MFMAs.
//      A query with no unmasked key gets O = 0.
#include <type_traits>

#include "device_common.h"
#include "kernels.h"

namespace rmm {

namespace {

namespace attk {
constexpr int NW = 8, NT = NW * 64;        // waves (32 queries each), threads
constexpr int BQ = NW * 32;                // queries per workgroup
constexpr int CNT = 256;                   // threads of the key-compaction kernel
constexpr int BN = 64;                     // keys per tile
constexpr int D = 128;                     // head dim (Q, K and V rows)
constexpr int RW = D / 2 + 1;              // words per staged Q / K row (odd)
constexpr int CH = D / 8;                  // 16-byte chunks per Q / K / V row
constexpr int VROW = D * 2;                // bytes per staged V row
constexpr int VTILE = BN * VROW;           // bytes of V per slot
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kTau = 8.f;                // lazy-rescale threshold, log2 units
constexpr uint32_t kOut = 0x80000000u;     // buffer offset past any range: reads zeros
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));

// One ring slot: 64 key rows of 2*KS data chunks + 1 pad chunk (an odd count
// of 16-byte chunks per row, so 8 or 16 consecutive rows at one chunk fall on
// distinct banks), then 64 V rows, then 1 KB that absorbs the wave-uniform
// padding of the key DMA.
template <int KS> constexpr int ktile_bytes() { return BN * (2 * KS + 1) * 16; }
template <int KS> constexpr int junk_offset() { return ktile_bytes<KS>() + VTILE; }
template <int KS> constexpr int slot_bytes() { return junk_offset<KS>() + 1024; }
// a slot also holds half of the block's Q rows (odd row stride) before the ring starts
constexpr int QHALF_BYTES = BQ / 2 * RW * 4;
template <int KS> constexpr int ring_slot_bytes() {
    return ((slot_bytes<KS>() > QHALF_BYTES ? slot_bytes<KS>() : QHALF_BYTES) + 1023) / 1024 * 1024;
}

// s_waitcnt vmcnt(N), expcnt and lgkmcnt unconstrained
template <int N>
__device__ __forceinline__ void wait_vmcnt_le() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
}

// x of lane l combined with x of lane l ^ 32 (both lanes get the result)
__device__ __forceinline__ float pair_max(float x) {
#if defined(__HIP_DEVICE_COMPILE__)
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
#else
    return x;
#endif
}
__device__ __forceinline__ float pair_sum(float x) {
#if defined(__HIP_DEVICE_COMPILE__)
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
#else
    return x;
#endif
}
}  // namespace attk

// Ki[bh][t][j] = K[b][g][t][I_h[j]] for j < k, 0 for k <= j < 16*KS.
template <int KS>
__global__ __launch_bounds__(attk::CNT) void attn_compact_k_kernel(
    const uint16_t *__restrict__ Kc, const int32_t *__restrict__ idx, uint16_t *__restrict__ Ki,
    int H, int Hkv, int Lk, int k) {
    using namespace attk;
    constexpr int KP = 16 * KS, CPR = 2 * KS;
    __shared__ uint32_t rows_lds[BN * RW];
    __shared__ uint16_t col_off[KP];
    const int tid = threadIdx.x;
    const int bh = blockIdx.y, b = bh / H, h = bh % H, g = h / (H / Hkv);
    const int t0 = blockIdx.x * BN;
    const int rows = min(BN, Lk - t0);
    const int32_t *I = idx + static_cast<int64_t>(bh) * k;
    for (int j = tid; j < KP; j += CNT) col_off[j] = static_cast<uint16_t>((j < k ? I[j] : D) * 2);
    for (int r = tid; r < BN; r += CNT) rows_lds[r * RW + D / 2] = 0u;
    const __amdgpu_buffer_rsrc_t kr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t *>(Kc + ((static_cast<int64_t>(b) * Hkv + g) * Lk + t0) * D), 0,
        static_cast<uint32_t>(rows * D * 2), 0x00020000);
#pragma unroll
    for (int i = 0; i < BN * CH / CNT; ++i) {
        const int v = tid + CNT * i;
        const auto x = __builtin_amdgcn_raw_buffer_load_b128(kr, static_cast<uint32_t>(v * 16), 0, 0);
        uint32_t *dst = rows_lds + (v / CH) * RW + (v % CH) * 4;
        dst[0] = x[0]; dst[1] = x[1]; dst[2] = x[2]; dst[3] = x[3];
    }
    __syncthreads();
    uint16_t *out = Ki + (static_cast<int64_t>(bh) * Lk + t0) * KP;
    for (int i = tid; i < rows * CPR; i += CNT) {
        const int r = i / CPR, cc = i % CPR;
        const char *base = reinterpret_cast<const char *>(rows_lds + r * RW);
        uint32_t w[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const uint32_t lo = *reinterpret_cast<const uint16_t *>(base + col_off[8 * cc + 2 * q]);
            const uint32_t hi = *reinterpret_cast<const uint16_t *>(base + col_off[8 * cc + 2 * q + 1]);
            w[q] = lo | (hi << 16);
        }
        *reinterpret_cast<uint4 *>(out + r * KP + 8 * cc) = make_uint4(w[0], w[1], w[2], w[3]);
    }
}

// KM selects the output form.  false: O[b][h][q][d].  true: the block output
// as the K-major input of the projection that follows attention (heads
// concatenated along its contraction axis), Ot[b][h*D + d][q] with row stride
// ldot, plus part[b][qt][h*D + d] = sum over the block's queries q < Lq of
// bf16(O[q][d])^2 in float64 (one query tile's share of that input's column
// energies; a fixed-order sum over the tiles completes them).
template <int KS, bool KM>
__global__ __launch_bounds__(attk::NT, 1) void attn_fwd_kernel(
    const uint16_t *__restrict__ Q, const uint16_t *__restrict__ Ki,
    const uint16_t *__restrict__ V, const int32_t *__restrict__ idx, uint16_t *__restrict__ O,
    int H, int Hkv, int Lq, int Lk, int k, float c, int neg_q, int causal, int64_t ldot,
    double *__restrict__ part) {
    using namespace attk;
    constexpr int KP = 16 * KS;                 // Ki row width
    constexpr int KRB = KP * 2;                 // Ki row bytes
    constexpr int KSL = 2 * KS + 1;             // 16-byte LDS chunks per staged key row
    constexpr int NJK = KSL;                    // DMA wave-instructions per key tile
    constexpr int PER_K = (NJK + NW - 1) / NW;  // per wave (the surplus lands in the junk area)
    constexpr int VPW = VTILE / 1024 / NW;      // V DMA wave-instructions per wave
    constexpr int PER = PER_K + VPW;            // DMA instructions per wave per tile
    constexpr int SB = ring_slot_bytes<KS>();
    static_assert(VPW * NW * 1024 == VTILE, "V tile split");

    __shared__ __attribute__((aligned(1024))) char slot0[SB];
    __shared__ __attribute__((aligned(1024))) char slot1[SB];
    __shared__ __attribute__((aligned(1024))) char slot2[SB];   // Q rows 0..127 before the ring
    __shared__ __attribute__((aligned(1024))) char slot3[SB];   // Q rows 128..255 before the ring
    __shared__ __attribute__((aligned(16))) uint16_t col_off[KP];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lr = lane & 31, lh = lane >> 5;
    const int nq = (Lq + BQ - 1) / BQ;
    const int BH = static_cast<int>(gridDim.x) / nq;
    // Work order: query tiles with the most key tiles first (causal).  When
    // the head count is a multiple of 8, the XCD that receives workgroup
    // `lin` (workgroups are dealt to the 8 XCDs in turn) gets a contiguous
    // range of heads, so heads that share a kv head share its L2.
    const int lin = blockIdx.x;
    int bh, rank;
    if (BH % 8 == 0) {
        const int hpx = BH / 8, j = lin / 8;
        bh = (lin % 8) * hpx + j % hpx;
        rank = j / hpx;
    } else {
        bh = lin % BH;
        rank = lin / BH;
    }
    const int b = bh / H, h = bh % H, g = h / (H / Hkv);
    const int qt = causal ? nq - 1 - rank : rank;
    const int q0 = qt * BQ;
    const int off = Lk - Lq;
    int n_tiles = (Lk + BN - 1) / BN;
    if (causal) {
        const int limit = min(q0 + BQ, Lq) - 1 + off;
        n_tiles = limit < 0 ? 0 : min(n_tiles, limit / BN + 1);
    }
    const int lend = min(Lk, n_tiles * BN);     // no row of the block keeps a key at or past this

    const int32_t *I = idx + static_cast<int64_t>(bh) * k;
    for (int j = tid; j < KP; j += NT) col_off[j] = static_cast<uint16_t>((j < k ? I[j] : D) * 2);

    // ---- DMA addressing (per lane, the same for every tile)
    uint32_t ksrc[PER_K], vsrc[VPW];
#pragma unroll
    for (int u = 0; u < PER_K; ++u) {
        const int j = wave + NW * u, i = 64 * j + lane;
        const int r = i / KSL, cc = i % KSL;
        ksrc[u] = (j < NJK && cc < 2 * KS) ? static_cast<uint32_t>(r * KRB + 16 * cc) : kOut;
    }
#pragma unroll
    for (int u = 0; u < VPW; ++u) {
        // V row chunk p of row r goes to LDS chunk p ^ 4*(r % 4) (r % 4 == lane / 16)
        const int j = wave + NW * u, r = 4 * j + (lane >> 4), p = lane & 15;
        vsrc[u] = static_cast<uint32_t>(r * VROW + 16 * (p ^ (4 * (lane >> 4))));
    }
    const uint16_t *Kih = Ki + static_cast<int64_t>(bh) * Lk * KP;
    const uint16_t *Vh = V + (static_cast<int64_t>(b) * Hkv + g) * Lk * D;
    auto dma = [&](char *slot, int kt) __attribute__((always_inline)) {
        const int t0 = __builtin_amdgcn_readfirstlane(min(kt * BN, Lk));
        const int rows = __builtin_amdgcn_readfirstlane(max(0, min(BN, lend - t0)));
        const __amdgpu_buffer_rsrc_t kr = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint16_t *>(Kih + static_cast<int64_t>(t0) * KP), 0,
            static_cast<uint32_t>(rows * KRB), 0x00020000);
        const __amdgpu_buffer_rsrc_t vr = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint16_t *>(Vh + static_cast<int64_t>(t0) * D), 0,
            static_cast<uint32_t>(rows * VROW), 0x00020000);
#pragma unroll
        for (int u = 0; u < PER_K; ++u) {
            const int j = wave + NW * u;
            lds_load16(kr, slot + (j < NJK ? 1024 * j : junk_offset<KS>()), ksrc[u]);
        }
#pragma unroll
        for (int u = 0; u < VPW; ++u)
            lds_load16(vr, slot + ktile_bytes<KS>() + 1024 * (wave + NW * u), vsrc[u]);
    };

    // ---- Q: read the block's rows, start the first two key tiles, stage Q
    //      (rows 0..127 in slot 2, 128..255 in slot 3), gather this wave's
    //      retained dims
    {
        constexpr int QPT = BQ * CH / NT;       // 16-byte chunks per thread; chunk i is row tid/16 + 32 i
        const __amdgpu_buffer_rsrc_t qr = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint16_t *>(Q + (static_cast<int64_t>(bh) * Lq + q0) * D), 0,
            static_cast<uint32_t>(min(BQ, Lq - q0) * D * 2), 0x00020000);
        uint4 rq[QPT];
#pragma unroll
        for (int i = 0; i < QPT; ++i) {
            const auto x = __builtin_amdgcn_raw_buffer_load_b128(qr, static_cast<uint32_t>((tid + NT * i) * 16), 0, 0);
            rq[i] = make_uint4(x[0], x[1], x[2], x[3]);
        }
        dma(slot0, 0);
        dma(slot1, 1);
        if (tid < 128) reinterpret_cast<uint32_t *>(slot2)[tid * RW + D / 2] = 0u;
        else if (tid < 256) reinterpret_cast<uint32_t *>(slot3)[(tid - 128) * RW + D / 2] = 0u;
#pragma unroll
        for (int i = 0; i < QPT; ++i) {
            const int v = tid + NT * i, r = v / CH;
            uint32_t *dst = reinterpret_cast<uint32_t *>(i < QPT / 2 ? slot2 : slot3) +
                            (r % 128) * RW + (v % CH) * 4;
            dst[0] = rq[i].x; dst[1] = rq[i].y; dst[2] = rq[i].z; dst[3] = rq[i].w;
        }
    }
    lds_barrier();
    bf16x8_t qf[KS];
    {
        const uint32_t flip = neg_q ? 0x80008000u : 0u;   // exact negation, for scale < 0
        const int row = wave * 32 + lr;
        const char *base = reinterpret_cast<const char *>(
            reinterpret_cast<const uint32_t *>(wave < NW / 2 ? slot2 : slot3) + (row % 128) * RW);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const uint4 co = *reinterpret_cast<const uint4 *>(&col_off[ks * 16 + 8 * lh]);
            const uint32_t o[4] = {co.x, co.y, co.z, co.w};
            uint32_t w[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint32_t lo = *reinterpret_cast<const uint16_t *>(base + (o[q] & 0xffffu));
                const uint32_t hi = *reinterpret_cast<const uint16_t *>(base + (o[q] >> 16));
                w[q] = (lo | (hi << 16)) ^ flip;
            }
            qf[ks] = __builtin_bit_cast(bf16x8_t, make_uint4(w[0], w[1], w[2], w[3]));
        }
    }

    // ---- per-lane fragment addressing
    // K fragment (A of S^T): key row 32*tb + lane%32, chunk 2*ks + lane/32
    const int kaddr = (lr * KSL + lh) * 16;
    // V^T fragment (A of O^T): 16-lane group gr reads keys 16*st + 4*(gr/2) + s16/4
    // (and +8) of dims 32*db + 16*(gr%2) + 4*(s16%4) .. +3 (transposing read)
    const int gr = lane >> 4, s16 = lane & 15, vv = s16 >> 2, qq = s16 & 3;
    int voff[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
        voff[db] = ktile_bytes<KS>() + (4 * (gr >> 1) + vv) * VROW +
                   ((4 * (db ^ vv) + 2 * (gr & 1) + (qq >> 1)) * 16) + 8 * (qq & 1);

    f32x16_t o_acc[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) o_acc[db][v] = 0.f;
    float m_run = -__builtin_inff(), l_run = 0.f;
    const int qw0 = q0 + wave * 32;
    const int lim = causal ? min(qw0 + lr + off, Lk - 1) : Lk - 1;          // this lane's query keeps keys <= lim
    const int lim_lo = causal ? min(qw0 + off, Lk - 1) : Lk - 1;           // every row of the wave keeps these
    const int lim_hi = causal ? min(qw0 + 31 + off, Lk - 1) : Lk - 1;      // no row of the wave keeps a key above

    // scores of the tile last multiplied, and weights waiting for their PV
    f32x16_t s[2];
    bf16x8_t pf[BN / 16];
    // S^T of tile kt: s[tb][v] is key kt*BN + 32*tb + 8*(v/4) + 4*lh + v%4 of query qw0 + lr
    auto qk = [&](const char *slot) __attribute__((always_inline)) {
        // all of the tile's fragments are read first, so the MFMAs wait once
        bf16x8_t kf[KS][2];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
            for (int tb = 0; tb < 2; ++tb)
                kf[ks][tb] = *reinterpret_cast<const bf16x8_t *>(slot + kaddr + (32 * tb * KSL + 2 * ks) * 16);
        __builtin_amdgcn_sched_barrier(0);       // keep the reads ahead of the MFMAs
#pragma unroll
        for (int tb = 0; tb < 2; ++tb)
#pragma unroll
            for (int v = 0; v < 16; ++v) s[tb][v] = 0.f;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
            for (int tb = 0; tb < 2; ++tb)
                s[tb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[ks][tb], qf[ks], s[tb], 0, 0, 0);
    };
    auto softmax = [&](int kt) __attribute__((always_inline)) {
        const int t0 = kt * BN;
        float mx = -__builtin_inff();
        if (t0 + BN - 1 > lim_lo) {              // the tile crosses some row's limit
            const int rel = lim - t0 - 4 * lh;   // key t0 + 4*lh + x is kept iff x <= rel
#pragma unroll
            for (int tb = 0; tb < 2; ++tb)
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    if (32 * tb + 8 * (v >> 2) + (v & 3) > rel) s[tb][v] = -__builtin_inff();
        }
        {
            // four independent chains, then combined
            float m4[4] = {-__builtin_inff(), -__builtin_inff(), -__builtin_inff(), -__builtin_inff()};
#pragma unroll
            for (int tb = 0; tb < 2; ++tb)
#pragma unroll
                for (int v = 0; v < 16; ++v) m4[v & 3] = fmaxf(m4[v & 3], s[tb][v]);
            mx = fmaxf(fmaxf(m4[0], m4[1]), fmaxf(m4[2], m4[3]));
        }
        mx = pair_max(mx);
        const float mt = mx == -__builtin_inff() ? -__builtin_inff() : mx * c;
        const bool need = mt > m_run + kTau;
        if (__builtin_amdgcn_ballot_w64(need)) {
            const float alpha = need ? __builtin_amdgcn_exp2f(m_run - mt) : 1.f;
            l_run *= alpha;
#pragma unroll
            for (int db = 0; db < D / 32; ++db)
#pragma unroll
                for (int v = 0; v < 16; ++v) o_acc[db][v] *= alpha;
            m_run = need ? mt : m_run;
        }
        // a row with nothing kept yet has only masked (-inf) scores here
        const float mu = m_run == -__builtin_inff() ? 0.f : m_run;
        float l4[4] = {0.f, 0.f, 0.f, 0.f};      // four independent chains
#pragma unroll
        for (int tb = 0; tb < 2; ++tb)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(s[tb][v], c, -mu));
                s[tb][v] = p;
                l4[v & 3] += p;
            }
        l_run += (l4[0] + l4[1]) + (l4[2] + l4[3]);
        // weights of keys 16*st + 8*(e/4) + 4*lh + e%4: the k-slot order of the V^T fragments
#pragma unroll
        for (int st = 0; st < BN / 16; ++st) {
            const int tb = st >> 1, g0 = 2 * (st & 1);
#pragma unroll
            for (int e = 0; e < 8; ++e) pf[st][e] = static_cast<__bf16>(s[tb][4 * (g0 + (e >> 2)) + (e & 3)]);
        }
    };
    auto pv = [&](const char *slot) __attribute__((always_inline)) {
        // all of the tile's V^T fragments are read first, so the MFMAs wait once
        bf16x8_t vf[BN / 16][D / 32];
#pragma unroll
        for (int st = 0; st < BN / 16; ++st)
#pragma unroll
            for (int db = 0; db < D / 32; ++db) {
                const char *p = slot + voff[db] + 16 * st * VROW;
                const s16x4_t lo = lds_read_tr16(p);
                const s16x4_t hi = lds_read_tr16(p + 8 * VROW);
                vf[st][db] = __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
            }
        __builtin_amdgcn_sched_barrier(0);       // keep the reads ahead of the MFMAs
#pragma unroll
        for (int st = 0; st < BN / 16; ++st)
#pragma unroll
            for (int db = 0; db < D / 32; ++db)
                o_acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[st][db], pf[st], o_acc[db], 0, 0, 0);
    };

    // ---- the ring.  Tile kt lives in slot kt % 4 and is loaded two steps
    // ahead.  Step i multiplies the keys of tile i (QK) and the values of tile
    // i-1 (PV).  The two halves of the workgroup (one wave of each per SIMD)
    // run the softmax at opposite ends of the step: the first half does
    // PV(i-1), QK(i), softmax(i); the second softmax(i-1), PV(i-1), QK(i).
    // So while one wave of a SIMD is in its exp/max work the other is in its
    // MFMAs.  Every step issues one tile of loads (tiles past the block's last
    // one read nothing and stage zeros), so the wait before each barrier is a
    // fixed vmcnt: the tile after the next may stay in flight.
    wait_vmcnt_le<PER>();
    lds_barrier();                               // tile 0 landed; Q gathered by every wave
    auto slot_ptr = [&](auto S) -> char * {
        constexpr int sl = decltype(S)::value;
        if constexpr (sl == 0) return slot0;
        else if constexpr (sl == 1) return slot1;
        else if constexpr (sl == 2) return slot2;
        else return slot3;
    };
    const bool late = wave >= NW / 2;
    // a tile with work for this wave: in range and not wholly masked for its rows
    auto active = [&](int kt) { return kt >= 0 && kt < n_tiles && kt * BN <= lim_hi; };
    auto step = [&](auto S, int i) __attribute__((always_inline)) {
        constexpr int sl = decltype(S)::value;
        dma(slot_ptr(std::integral_constant<int, (sl + 2) % 4>{}), i + 2);
        const bool prev = active(i - 1), cur = active(i);
        if (late && prev) softmax(i - 1);
        if (prev) pv(slot_ptr(std::integral_constant<int, (sl + 3) % 4>{}));
        if (cur) qk(slot_ptr(S));
        if (!late && cur) softmax(i);
        wait_vmcnt_le<PER>();
        lds_barrier();
    };
    for (int i = 0; i <= n_tiles; i += 4) {
        step(std::integral_constant<int, 0>{}, i);
        step(std::integral_constant<int, 1>{}, i + 1);
        step(std::integral_constant<int, 2>{}, i + 2);
        step(std::integral_constant<int, 3>{}, i + 3);
    }
    wait_vmcnt_le<0>();                          // the trailing out-of-range loads

    const float l = pair_sum(l_run);
    const float inv = l > 0.f ? 1.f / l : 0.f;
    const int ql = wave * 32 + lr;               // rows past Lq fall outside the buffer
    if constexpr (KM) {
        // ---- O^T of the block through the idle ring: dim d in slot d / 64, row
        //      d % 64 (OROW bytes: 256 queries + a 16-byte pad, so the two lane
        //      halves, 4 dims apart, write distinct banks), query column ql
        constexpr int OROW = BQ * 2 + 16;
        static_assert(64 * OROW <= SB, "staged O^T rows");
        __syncthreads();                         // every wave's last reads and loads are done
#pragma unroll
        for (int db = 0; db < D / 32; ++db) {
            char *so = (db < 2 ? slot0 : slot1) + (32 * (db & 1) + 4 * lh) * OROW + 2 * ql;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const __bf16 x = static_cast<__bf16>(o_acc[db][v] * inv);
                *reinterpret_cast<__bf16 *>(so + (8 * (v >> 2) + (v & 3)) * OROW) = x;
            }
        }
        __syncthreads();
        const int nvq = min(BQ, Lq - q0);           // queries of the block (Lq % 8 == 0)
        // stores: each half-wave writes one dim row per pass, 32 lanes x 16
        // bytes = the block's 256 queries
        {
            const int cq = lane & 31, rr = tid >> 5;     // rr = 0..15
            uint16_t *Otb = O + (static_cast<int64_t>(b) * H + h) * D * ldot + q0;
#pragma unroll
            for (int i = 0; i < D / 16; ++i) {
                const int dd = rr + 16 * i;
                const uint4 w = *reinterpret_cast<const uint4 *>((i < 4 ? slot0 : slot1) + (dd & 63) * OROW + 16 * cq);
                if (8 * cq < nvq) *reinterpret_cast<uint4 *>(Otb + dd * ldot + 8 * cq) = w;
            }
        }
        // energies: thread t sums dim row t/4 over its quarter of the queries
        // (64, as eight 16-byte pieces), then the quad adds its four quarters
        // (lane ^ 1, then lane ^ 2: every lane of the quad ends with the same sum)
        {
            const int dd = tid >> 2, qa = tid & 3;
            const char *row = (dd < 64 ? slot0 : slot1) + (dd & 63) * OROW;
            double e = 0.0;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int ch = 8 * qa + j;
                if (8 * ch < nvq) {
                    const uint4 w = *reinterpret_cast<const uint4 *>(row + 16 * ch);
                    const uint32_t u[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const double lo = static_cast<double>(__uint_as_float(u[q] << 16));
                        const double hi = static_cast<double>(__uint_as_float(u[q] & 0xffff0000u));
                        e = fma(lo, lo, e);
                        e = fma(hi, hi, e);
                    }
                }
            }
            e += dpp_f64<0xB1>(e);
            e += dpp_f64<0x4E>(e);
            if (qa == 0)
                part[(static_cast<int64_t>(b) * nq + qt) * H * D + static_cast<int64_t>(h) * D + dd] = e;
        }
        return;
    }
    // ---- O[q][d]: the lane holds d = 32*db + 8*gq + 4*lh + {0..3} of query qw0 + lr
    const __amdgpu_buffer_rsrc_t orr = __builtin_amdgcn_make_buffer_rsrc(
        O + (static_cast<int64_t>(bh) * Lq + q0) * D, 0,
        static_cast<uint32_t>(min(BQ, Lq - q0) * D * 2), 0x00020000);
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int gq = 0; gq < 4; ++gq) {
            const uint32_t w0 = pack_bf16x2(o_acc[db][4 * gq] * inv, o_acc[db][4 * gq + 1] * inv);
            const uint32_t w1 = pack_bf16x2(o_acc[db][4 * gq + 2] * inv, o_acc[db][4 * gq + 3] * inv);
            __builtin_amdgcn_raw_buffer_store_b64(
                u32x2_t{w0, w1}, orr, static_cast<uint32_t>((ql * D + 32 * db + 8 * gq + 4 * lh) * 2), 0, 0);
        }
}

template <int KS, bool KM>
hipError_t launch_ks(const uint16_t *Q, const uint16_t *Kc, const uint16_t *V, const int32_t *idx,
                     int64_t batch, int64_t H, int64_t Hkv, int64_t Lq, int64_t Lk, int64_t k,
                     float scale, bool causal, uint16_t *O, uint16_t *Ki, int64_t ldot,
                     double *part, hipStream_t stream) {
    using namespace attk;
    const unsigned BH = static_cast<unsigned>(batch * H);
    hipLaunchKernelGGL(attn_compact_k_kernel<KS>, dim3(static_cast<unsigned>((Lk + BN - 1) / BN), BH),
                       dim3(CNT), 0, stream, Kc, idx, Ki, static_cast<int>(H), static_cast<int>(Hkv),
                       static_cast<int>(Lk), static_cast<int>(k));
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const unsigned nq = static_cast<unsigned>((Lq + BQ - 1) / BQ);
    // |scale| in log2 units; a zero scale is applied as the smallest normal
    // float, which leaves every finite score's weight exactly 1 (as zero
    // would) while masked -inf scores still give weight 0
    float c = (scale < 0.f ? -scale : scale) * kLog2e;
    if (c < 1.17549435e-38f) c = 1.17549435e-38f;
    hipLaunchKernelGGL((attn_fwd_kernel<KS, KM>), dim3(nq * BH), dim3(NT), 0, stream,
                       Q, Ki, V, idx, O, static_cast<int>(H), static_cast<int>(Hkv),
                       static_cast<int>(Lq), static_cast<int>(Lk), static_cast<int>(k), c,
                       scale < 0.f ? 1 : 0, causal ? 1 : 0, ldot, part);
    return hipGetLastError();
}

template <bool KM>
hipError_t launch_attn(const uint16_t *Q, const uint16_t *Kc, const uint16_t *V,
                       const int32_t *idx, int64_t batch, int64_t H, int64_t Hkv, int64_t Lq,
                       int64_t Lk, int64_t k, float scale, bool causal, uint16_t *O, uint16_t *Ki,
                       int64_t ldot, double *part, hipStream_t stream) {
    switch (attn_k_steps(k)) {
    case 2: return launch_ks<2, KM>(Q, Kc, V, idx, batch, H, Hkv, Lq, Lk, k, scale, causal, O, Ki, ldot, part, stream);
    case 4: return launch_ks<4, KM>(Q, Kc, V, idx, batch, H, Hkv, Lq, Lk, k, scale, causal, O, Ki, ldot, part, stream);
    case 6: return launch_ks<6, KM>(Q, Kc, V, idx, batch, H, Hkv, Lq, Lk, k, scale, causal, O, Ki, ldot, part, stream);
    default: return launch_ks<8, KM>(Q, Kc, V, idx, batch, H, Hkv, Lq, Lk, k, scale, causal, O, Ki, ldot, part, stream);
    }
}

}  // namespace

int attn_k_steps(int64_t k) { return k <= 32 ? 2 : k <= 64 ? 4 : k <= 96 ? 6 : 8; }

size_t attn_workspace_bytes(int64_t batch_heads, int64_t Lk, int64_t k) {
    return static_cast<size_t>(batch_heads) * static_cast<size_t>(Lk) *
           static_cast<size_t>(16 * attn_k_steps(k)) * 2;
}

int64_t attn_query_tiles(int64_t Lq) { return (Lq + attk::BQ - 1) / attk::BQ; }

hipError_t launch_attn_bf16(const uint16_t *Q, const uint16_t *Kc, const uint16_t *V,
                            const int32_t *idx, int64_t batch, int64_t H, int64_t Hkv,
                            int64_t Lq, int64_t Lk, int64_t k, float scale, bool causal,
                            uint16_t *O, void *workspace, hipStream_t stream) {
    return launch_attn<false>(Q, Kc, V, idx, batch, H, Hkv, Lq, Lk, k, scale, causal, O,
                              static_cast<uint16_t *>(workspace), 0, nullptr, stream);
}

hipError_t launch_attn_kmajor_bf16(const uint16_t *Q, const uint16_t *Kc, const uint16_t *V,
                                   const int32_t *idx, int64_t batch, int64_t H, int64_t Hkv,
                                   int64_t Lq, int64_t Lk, int64_t k, float scale, bool causal,
                                   uint16_t *Ot, int64_t ldot, double *energy, uint16_t *Ki,
                                   double *partials, hipStream_t stream) {
    const hipError_t e = launch_attn<true>(Q, Kc, V, idx, batch, H, Hkv, Lq, Lk, k, scale, causal,
                                           Ot, Ki, ldot, partials, stream);
    if (e != hipSuccess) return e;
    // energies: the query tiles' partial sums, added in tile order
    return launch_score_finalize(partials, batch, attn_query_tiles(Lq), H * attk::D, energy, stream);
}

}  // namespace rmm
