// Decode products of B sequences over the union of their retained sets
// (Sec. 3.2 definition of RMM; App. A: during decoding each sequence's set
// follows its own current token).
//
//   Y[b][n] = sum_{t < k} X[b][I_b[t]] * W[I_b[t]][n],   b < B <= 32
//
// The per-sequence product reads k rows of W for every sequence (B*k*N*2
// bytes), more than the whole of W once B*r > 1.  Here every row that some
// sequence keeps is read once: over the union U of the B sets,
//
//   Y[b][n] = sum_{j in U} xs[b][j] * W[j][n],   xs[b][j] = X[b][j] if j in
//                                                 I_b, else 0,
//
// a product of a B x |U| matrix with |U| rows of W, done on the MFMA units
// (32 sequences x 32 columns per v_mfma_f32_32x32x16_bf16).  For finite W
// each sequence's sum has exactly the terms of its own set (the others are
// exact zeros); the order of the additions differs from the per-sequence
// kernel, so results agree within rounding, not bit for bit.
//
// The contraction axis is cut into ranges of kShareRange indices.  Four
// launches:
//   1. share_offsets_kernel: for every sequence and range boundary, the first
//      position of the sequence's (ascending) list at or past it -- each list
//      position writes the boundaries between its predecessor and itself, so
//      every entry has one writer and no memory needs clearing;
//   2. share_union_kernel, one workgroup per range: the sequences'
//      activations over the range are staged in LDS, the members of each
//      sequence's sub-list set bits of a per-index sequence mask in LDS
//      (atomic OR: order-free), the indices with a nonzero mask are compacted
//      in ascending order (a block scan), and the range's union rows and
//      xs[b][row] (bf16, zeros past the union and for sequences that do not
//      keep the row) go to the workspace;
//   3. share_product_kernel, one workgroup per (range, column chunk: 128
//      columns below eight sequences, 256 from eight on): the union rows of
//      W stream through an LDS ring by LDS DMA (six slots of 32 rows, or
//      four of the wider rows), W fragments come back with the
//      transposing LDS read, xs fragments are loaded into registers with
//      their stage; each range writes fp32 partials (or Y when there is one
//      range);
//   4. share_reduce_kernel adds the ranges' partials in range order.
#include <type_traits>
#include <utility>

#include "device_common.h"
#include "kernels.h"
#include "gemv_shared.h"

namespace rmm {

namespace {

namespace sh {
constexpr int RG = kShareRange;    // contraction indices per range
constexpr int NT = 256;            // threads of every kernel here
constexpr int NW = NT / 64;
constexpr int RS = 32;             // union rows per stage
}  // namespace sh

// Product tile by batch size: 128 columns and six ring slots for fewer than
// eight sequences (small unions: more, shorter workgroups), 256 columns
// (512-byte staged rows) and four slots from eight on.
constexpr int kShareWideB = 8;
inline int share_cols(int64_t B) { return B >= kShareWideB ? 256 : 128; }

// s_waitcnt vmcnt(N) with expcnt and lgkmcnt unconstrained
template <int N>
__device__ __forceinline__ void share_wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
}

// group of workgroup `bid` in a launch whose groups start at first(g)
template <typename F>
__device__ __forceinline__ int share_group(const ShareGroups &G, int bid, F first) {
    int g = 0;
    while (g + 1 < G.n && bid >= first(G.g[g + 1])) ++g;
    return g;
}

// 1. list positions of the range boundaries: pos[b][r] = first t with
// I_b[t] >= r * RG (pos[b][R] = k)
__global__ __launch_bounds__(sh::NT) void share_offsets_kernel(ShareGroups G, int B) {
    const int bid = static_cast<int>(blockIdx.x);
    const int gi = share_group(G, bid, [](const ShareGroup &q) { return q.first_o; });
    const ShareGroup &q = G.g[gi];
    const int per = (q.k + sh::NT - 1) / sh::NT;     // workgroups per sequence
    const int local = bid - q.first_o;
    const int b = local / per;
    const int t = (local % per) * sh::NT + static_cast<int>(threadIdx.x);
    if (b >= B || t >= q.k) return;
    const int32_t *I = q.idx + static_cast<int64_t>(b) * q.k;
    int32_t *pos = q.pos + static_cast<int64_t>(b) * (q.R + 1);
    // indices outside [0, K) are clamped (lists are required to lie within it)
    auto range_of = [&](int32_t j) { return min(max(j, 0), q.K - 1) / sh::RG; };
    const int hi = range_of(I[t]);
    const int lo = t == 0 ? -1 : range_of(I[t - 1]);
    for (int r = lo + 1; r <= hi; ++r) pos[r] = t;
    if (t == q.k - 1)
        for (int r = hi + 1; r <= q.R; ++r) pos[r] = q.k;
}

// 2. the union of the B sub-lists of one range, and xs over it (1024
// threads: the work of one range is a few dependent LDS passes)
constexpr int kUnionThreads = 1024;
__global__ __launch_bounds__(kUnionThreads) void share_union_kernel(ShareGroups G, int B) {
    using namespace sh;
    constexpr int UT = kUnionThreads, UW = UT / 64;
    __shared__ uint32_t mask[RG];
    __shared__ int32_t lrow[RG];
    __shared__ uint32_t lmask[RG];
    __shared__ int32_t wsum[UW];
    __shared__ int32_t seg[kShareMaxB + 1];       // prefix sums of the sub-list lengths
    __shared__ int32_t beg[kShareMaxB];           // first list position of each sub-list
    __shared__ __attribute__((aligned(16))) uint16_t xr[kShareMaxB * RG];   // X over the range
    const int bid = static_cast<int>(blockIdx.x);
    const int gi = share_group(G, bid, [](const ShareGroup &q) { return q.first_u; });
    const ShareGroup &q = G.g[gi];
    const int r = bid - q.first_u;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int j0 = r * RG, nj = min(RG, q.K - j0);
    for (int i = tid; i < RG; i += UT) mask[i] = 0u;
    // the sub-lists of the range (clamped, so that a list that breaks the
    // ascending precondition still reads inside itself) and their offsets
    if (wave == 0) {
        int len = 0;
        if (lane < B) {
            const int32_t *pos = q.pos + static_cast<int64_t>(lane) * (q.R + 1);
            const int t0 = min(max(pos[r], 0), q.k);
            const int t1 = min(max(pos[r + 1], t0), q.k);
            beg[lane] = t0;
            len = t1 - t0;
        }
        int incl = len;
#pragma unroll
        for (int sft = 1; sft < 32; sft <<= 1) {
            const int v = __shfl_up(incl, sft);
            if (lane >= sft) incl += v;
        }
        if (lane < B) seg[lane + 1] = incl;
        if (lane == 0) seg[0] = 0;
    }
    // each sequence's activations over the range, 16 bytes at a time (X rows
    // are 16-byte aligned and j0 is a multiple of 8); past K: zeros, never kept
    const int cpr = RG / 8;
    for (int i = tid; i < B * cpr; i += UT) {
        const int b = i / cpr, c = i % cpr;
        const uint16_t *x = q.X + static_cast<int64_t>(b) * q.ldx + j0 + 8 * c;
        uint16_t *d = &xr[b * RG + 8 * c];
        if (8 * c + 8 <= nj) {
            *reinterpret_cast<uint4 *>(d) = *reinterpret_cast<const uint4 *>(x);
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) d[e] = 8 * c + e < nj ? x[e] : 0;
        }
    }
    __syncthreads();
    // every entry of every sub-list sets its sequence's bit (atomic OR:
    // order-free); entries are numbered across the sub-lists, four loads in
    // flight per thread
    const int E = seg[B];
    for (int e0 = tid; e0 < E; e0 += 4 * UT) {
        int jj[4];
        uint32_t bit[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int e = e0 + u * UT;
            jj[u] = -1;
            bit[u] = 0u;
            if (e < E) {
                int lo = 0, hi = B - 1;                // the sub-list holding entry e
                while (lo < hi) {
                    const int mid = (lo + hi + 1) >> 1;
                    if (seg[mid] <= e) lo = mid; else hi = mid - 1;
                }
                jj[u] = q.idx[static_cast<int64_t>(lo) * q.k + beg[lo] + (e - seg[lo])] - j0;
                bit[u] = 1u << lo;
            }
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
            if (jj[u] >= 0 && jj[u] < nj) atomicOr(&mask[jj[u]], bit[u]);
    }
    __syncthreads();
    // ascending compaction: thread tid < RG owns index tid
    const uint32_t m = tid < RG ? mask[tid] : 0u;
    const int c = m != 0u;
    int incl = c;                                  // inclusive scan within the wave
#pragma unroll
    for (int sft = 1; sft < 64; sft <<= 1) {
        const int v = __shfl_up(incl, sft);
        if (lane >= sft) incl += v;
    }
    if (lane == 63) wsum[wave] = incl;
    __syncthreads();
    int base = 0;
    for (int w = 0; w < wave; ++w) base += wsum[w];
    if (c) {
        lrow[base + incl - 1] = j0 + tid;
        lmask[base + incl - 1] = m;
    }
    int u = 0;
    for (int w = 0; w < UW; ++w) u += wsum[w];
    __syncthreads();
    const int up = (u + RS - 1) / RS * RS;
    int32_t *rows = q.rows + static_cast<int64_t>(r) * RG;
    for (int p = tid; p < u; p += UT) rows[p] = lrow[p];
    if (tid == 0) q.cnt[r] = u;
    // xs[r][b][p], p < up: the sequence's value where it keeps the row, two
    // rows per thread and store
    uint16_t *xs = q.xs + static_cast<int64_t>(r) * 32 * RG;
    const int hp = up / 2;
    for (int i = tid; i < B * hp; i += UT) {
        const int b = i / hp, p = 2 * (i % hp);
        uint32_t v = 0;
        if (p < u && ((lmask[p] >> b) & 1u)) v = xr[b * RG + lrow[p] - j0];
        if (p + 1 < u && ((lmask[p + 1] >> b) & 1u))
            v |= static_cast<uint32_t>(xr[b * RG + lrow[p + 1] - j0]) << 16;
        *reinterpret_cast<uint32_t *>(&xs[b * RG + p]) = v;
    }
}

// 3. the range's product for CW_ columns: Y^T tile (columns x sequences).
// The four waves take CW_/128 blocks of 32 columns each; the ring has NS_
// slots of 32 staged rows (NS_ - 1 stages in flight).
template <int N, typename F, int... I>
__device__ __forceinline__ void share_steps(F &&f, int st, int nst, std::integer_sequence<int, I...>) {
    static_assert(sizeof...(I) == N, "steps");
    ((st + I < nst ? f(std::integral_constant<int, I>{}, st + I) : void()), ...);
}

template <int CW_, int NS_>
__global__ __launch_bounds__(sh::NT, (160 * 1024) / (NS_ * sh::RS * CW_ * 2 + 4 * sh::RG + 1024))
void share_product_kernel(ShareGroups G, int B) {
    using namespace sh;
    constexpr int ROWB = CW_ * 2;              // bytes per staged W row
    constexpr int SLOT = RS * ROWB;            // bytes per ring slot
    constexpr int RPI = 1024 / ROWB;           // rows one wave instruction stages
    constexpr int LPR = ROWB / 16;             // lanes per staged row
    constexpr int PER = RS / RPI / NW;         // DMA instructions per wave per stage
    constexpr int NB = CW_ / 32 / NW;          // 32-column blocks per wave
    constexpr int DA = NS_ - 1;                // stages in flight ahead of the MFMAs
    constexpr int LPS = PER + RS / 16;         // vector loads per wave per stage (DMA + xs)
    static_assert(NB >= 1 && PER >= 1 && NS_ >= 3 && NS_ <= 8 && (DA - 1) * LPS < 64, "layout");
    __shared__ int32_t rl[RG];
    // one LDS object per ring slot: the compiler then sees that reading one
    // slot cannot alias the loads still landing in the others
    __shared__ __attribute__((aligned(1024))) char sl0[SLOT], sl1[SLOT], sl2[SLOT];
    __shared__ __attribute__((aligned(1024))) char sl3[NS_ > 3 ? SLOT : 16], sl4[NS_ > 4 ? SLOT : 16],
        sl5[NS_ > 5 ? SLOT : 16], sl6[NS_ > 6 ? SLOT : 16], sl7[NS_ > 7 ? SLOT : 16];
    auto slot_at = [&](auto I) -> char * {
        constexpr int i = decltype(I)::value;
        if constexpr (i == 0) return sl0;
        else if constexpr (i == 1) return sl1;
        else if constexpr (i == 2) return sl2;
        else if constexpr (i == 3) return sl3;
        else if constexpr (i == 4) return sl4;
        else if constexpr (i == 5) return sl5;
        else if constexpr (i == 6) return sl6;
        else return sl7;
    };
    const int bid = static_cast<int>(blockIdx.x);
    const int gi = share_group(G, bid, [](const ShareGroup &q) { return q.first_p; });
    const ShareGroup &q = G.g[gi];
    const int local = bid - q.first_p;
    const int r = local / q.chunks, chunk = local % q.chunks;
    const int n0 = chunk * CW_;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int u = min(max(q.cnt[r], 0), RG);      // written by the union kernel
    const int up = (u + RS - 1) / RS * RS;
    const int nst = up / RS;
    for (int p = tid; p < up; p += NT) rl[p] = p < u ? q.rows[static_cast<int64_t>(r) * RG + p] : 0;
    __syncthreads();

    // W rows from column n0 on; columns past N read padding or the next row
    // (never stored), rows past the matrix's end read zeros
    const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t *>(q.W + n0), 0,
        static_cast<uint32_t>((static_cast<int64_t>(q.K) * q.ldw - n0) * 2), 0x00020000);
    // the range's xs rows (sequences past B are never read)
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t *>(q.xs + static_cast<int64_t>(r) * 32 * RG), 0,
        static_cast<uint32_t>(32 * RG * 2), 0x00020000);
    const uint32_t wrow = static_cast<uint32_t>(q.ldw) * 2u;
    constexpr uint32_t kOut = 0x80000000u;
    // DMA role: instruction e of the wave stages rows RPI*(PER*wave + e) +
    // lane/LPR of a stage; the lane fills chunk position lane % LPR of its row
    // with source chunk (lane % LPR) ^ 4*(row % 4)
    const int drow = lane / LPR, dpos = lane % LPR;
    auto dma = [&](char *slot, int st) {
#pragma unroll
        for (int e = 0; e < PER; ++e) {
            const int row = RPI * (PER * wave + e);
            const int rr = row + drow;
            const int p = st * RS + rr;
            const uint32_t col = static_cast<uint32_t>(dpos ^ (4 * (rr & 3))) * 16u;
            const uint32_t off = p < u ? static_cast<uint32_t>(rl[p]) * wrow + col : kOut;
            lds_load16(wr, slot + row * ROWB, off);
        }
    };
    // xs fragment of a 16-row step (the MFMA's second operand): sequence
    // lane % 32, rows 8*(lane/32) .. +7, loaded into registers with the stage
    const int xb = lane & 31;
    const uint32_t xoff = static_cast<uint32_t>(xb * RG + 8 * (lane >> 5)) * 2u;
    bf16x8_t xq[NS_][RS / 16];
    auto xload = [&](bf16x8_t (&d)[RS / 16], int st) {
#pragma unroll
        for (int ks = 0; ks < RS / 16; ++ks) {
            const uint32_t off = xb < B && st < nst ? xoff + static_cast<uint32_t>(st * RS + ks * 16) * 2u : kOut;
            d[ks] = __builtin_bit_cast(bf16x8_t, __builtin_amdgcn_raw_buffer_load_b128(xr, off, 0, 0));
        }
    };
    // Fragment role (transposing read): 16-lane group g reads rows
    // 8*(g/2) + s/4 (+4) of a 16-row step, columns 16*(g%2) + 4*(s%4) .. +3 of
    // a 32-column block, whose 16-byte chunks sit at position ^ 4*(row % 4)
    const int g16 = lane >> 4, s16 = lane & 15;
    const int f4 = (s16 >> 2) & 3;
    const int col_off = (2 * (g16 & 1) + ((s16 & 3) >> 1)) * 16 + 8 * (s16 & 1);
    const int lane_off = (8 * (g16 >> 1) + (s16 >> 2)) * ROWB + col_off;
    int woff[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j) {
        const int qb = wave * NB + j;
        woff[j] = lane_off + 64 * ((qb & ~3) + ((qb & 3) ^ f4));
    }

    f32x16_t acc[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[j][v] = 0.f;
    // every step issues one stage of loads (past the last stage: out of
    // range, zeros into a slot or registers nobody reads), so the wait is a
    // fixed count
    auto issue = [&](auto I, int st) {
        dma(slot_at(I), st);
        xload(xq[decltype(I)::value], st);
    };
    share_steps<DA>([&](auto I, int st) { issue(I, st); }, 0, DA, std::make_integer_sequence<int, DA>{});
    share_wait_vmcnt<(DA - 1) * LPS>();
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_barrier" ::: "memory");
    // stage st lives in slot st % NS_; step st refills the slot read in step st - 1
    auto step = [&](auto I, int st) {
        constexpr int sl = decltype(I)::value, nx = (sl + DA) % NS_;
        issue(std::integral_constant<int, nx>{}, st + DA);
        const char *slot = slot_at(I);
#pragma unroll
        for (int ks = 0; ks < RS / 16; ++ks) {
#pragma unroll
            for (int j = 0; j < NB; ++j) {
                const char *wb = slot + woff[j] + ks * 16 * ROWB;
                const s16x4_t lo = lds_read_tr16(wb);
                const s16x4_t hi = lds_read_tr16(wb + 4 * ROWB);
                const bf16x8_t wf =
                    __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
                acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf, xq[sl][ks], acc[j], 0, 0, 0);
            }
        }
        share_wait_vmcnt<(DA - 1) * LPS>();       // stage st + 1 landed
        __builtin_amdgcn_sched_barrier(0);
        asm volatile("s_barrier" ::: "memory");
    };
    int st = 0;
    for (; st + NS_ <= nst; st += NS_) share_steps<NS_>(step, st, nst, std::make_integer_sequence<int, NS_>{});
    share_steps<NS_ - 1>(step, st, nst, std::make_integer_sequence<int, NS_ - 1>{});
    share_wait_vmcnt<0>();                          // the trailing out-of-range loads

    // acc[j][4*gq + i]: column n0 + 32*(wave*NB + j) + 8*gq + 4*(lane/32) + i,
    // sequence lane % 32
    const int b = lane & 31;
    if (b >= B) return;
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
        for (int gq = 0; gq < 4; ++gq)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int n = n0 + 32 * (wave * NB + j) + 8 * gq + 4 * (lane >> 5) + i;
                if (n >= q.N) continue;
                if (q.R == 1)
                    q.Y[static_cast<int64_t>(b) * q.ldy + n] = f32_to_bf16(acc[j][4 * gq + i]);
                else
                    q.P[(static_cast<int64_t>(b) * q.R + r) * q.N + n] = acc[j][4 * gq + i];
            }
}

// 4. Y[b][n] = the ranges' partials P[b][r][n] added in range order; a
// thread takes four consecutive columns of one sequence
__global__ __launch_bounds__(sh::NT) void share_reduce_kernel(ShareGroups G, int B) {
    const int bid = static_cast<int>(blockIdx.x);
    const int gi = share_group(G, bid, [](const ShareGroup &q) { return q.first_r; });
    const ShareGroup &q = G.g[gi];
    const int n4 = (q.N + 3) / 4;
    const int i = (bid - q.first_r) * sh::NT + static_cast<int>(threadIdx.x);
    if (q.R < 2 || i >= B * n4) return;
    const int b = i / n4, n = 4 * (i % n4);
    const float *p = q.P + static_cast<int64_t>(b) * q.R * q.N + n;
    float s[4] = {0.f, 0.f, 0.f, 0.f};
    if (q.N % 4 == 0) {
        int r = 0;
        for (; r + 8 <= q.R; r += 8) {
            float4 v[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = *reinterpret_cast<const float4 *>(p + static_cast<int64_t>(r + e) * q.N);
#pragma unroll
            for (int e = 0; e < 8; ++e) { s[0] += v[e].x; s[1] += v[e].y; s[2] += v[e].z; s[3] += v[e].w; }
        }
        for (; r < q.R; ++r) {
            const float4 v = *reinterpret_cast<const float4 *>(p + static_cast<int64_t>(r) * q.N);
            s[0] += v.x; s[1] += v.y; s[2] += v.z; s[3] += v.w;
        }
    } else {
        for (int r = 0; r < q.R; ++r)
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (n + e < q.N) s[e] += p[static_cast<int64_t>(r) * q.N + e];
    }
#pragma unroll
    for (int e = 0; e < 4; ++e)
        if (n + e < q.N) q.Y[static_cast<int64_t>(b) * q.ldy + n + e] = f32_to_bf16(s[e]);
}

}  // namespace

size_t share_group_layout(int64_t B, int64_t N, int64_t K, void *ws, ShareGroup *q) {
    auto a256 = [](size_t x) { return (x + 255) & ~static_cast<size_t>(255); };
    const int64_t R = (K + kShareRange - 1) / kShareRange;
    const size_t pos = a256(static_cast<size_t>(B * (R + 1)) * 4);
    const size_t rows = a256(static_cast<size_t>(R * kShareRange) * 4);
    const size_t cnt = a256(static_cast<size_t>(R) * 4);
    const size_t xs = a256(static_cast<size_t>(R * 32 * kShareRange) * 2);
    const size_t part = R > 1 ? a256(static_cast<size_t>(B * R * N) * 4) : 0;
    // addresses formed as integers: ws may be null when only the size is asked
    const uintptr_t p = reinterpret_cast<uintptr_t>(ws);
    q->pos = reinterpret_cast<int32_t *>(p);
    q->rows = reinterpret_cast<int32_t *>(p + pos);
    q->cnt = reinterpret_cast<int32_t *>(p + pos + rows);
    q->xs = reinterpret_cast<uint16_t *>(p + pos + rows + cnt);
    q->P = R > 1 ? reinterpret_cast<float *>(p + pos + rows + cnt + xs) : nullptr;
    q->R = static_cast<int>(R);
    q->chunks = static_cast<int>((N + share_cols(B) - 1) / share_cols(B));
    return pos + rows + cnt + xs + part;
}

hipError_t launch_share_products(ShareGroups G, int64_t B, hipStream_t stream) {
    int o = 0, un = 0, pr = 0, rd = 0;
    for (int i = 0; i < G.n; ++i) {
        ShareGroup &q = G.g[i];
        q.first_o = o;
        o += static_cast<int>(B) * ((q.k + sh::NT - 1) / sh::NT);
        q.first_u = un;
        un += q.R;
        q.first_p = pr;
        pr += q.R * q.chunks;
        q.first_r = rd;
        if (q.R > 1) rd += (static_cast<int>(B) * ((q.N + 3) / 4) + sh::NT - 1) / sh::NT;
    }
    const int Bi = static_cast<int>(B);
    hipLaunchKernelGGL(share_offsets_kernel, dim3(static_cast<unsigned>(o)), dim3(sh::NT), 0, stream, G, Bi);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(share_union_kernel, dim3(static_cast<unsigned>(un)), dim3(kUnionThreads), 0, stream,
                       G, Bi);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (share_cols(B) == 256)
        hipLaunchKernelGGL((share_product_kernel<256, 4>), dim3(static_cast<unsigned>(pr)), dim3(sh::NT), 0,
                           stream, G, Bi);
    else
        hipLaunchKernelGGL((share_product_kernel<128, 6>), dim3(static_cast<unsigned>(pr)), dim3(sh::NT), 0,
                           stream, G, Bi);
    if ((e = hipGetLastError()) != hipSuccess || rd == 0) return e;
    hipLaunchKernelGGL(share_reduce_kernel, dim3(static_cast<unsigned>(rd)), dim3(sh::NT), 0, stream, G, Bi);
    return hipGetLastError();
}

}  // namespace rmm
