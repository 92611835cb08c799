// TopK over each unit's energies (Sec. 3.2: I = TopK({s_j}, ceil(rho d))),
// returned as an ascending index list.
//
// One workgroup per selection unit.  Each float64 energy is mapped to a
// 64-bit key whose unsigned order is the order of the values (NaN above
// +inf, -0 == +0), so the whole selection is integer work: an MSB-first
// radix select with 8-bit digits finds the k-th largest key, using LDS
// histograms with integer atomics (order-independent counts).  It starts
// below the leading bits every key shares and stops as soon as the bucket
// holding the k-th key is taken whole.  Keys tied with
// the k-th key are taken lowest index first, and the kept indices are
// compacted in ascending order with two workgroup prefix scans.  Each thread
// owns a contiguous chunk of keys, kept in registers when it fits.  For a
// unit of one token (a decode step) the keys come straight from the token's
// activations: 16 (bf16) or 31 (fp32) key bits, so at most two passes.
#include "device_common.h"
#include "kernels.h"

namespace rmm {

namespace {

__device__ __forceinline__ uint64_t order_key(double d) {
    uint64_t u = __double_as_longlong(d);
    if (d != d) u = 0x7ff8000000000000ull;          // every NaN -> one quiet NaN
    if (u == 0x8000000000000000ull) u = 0;          // -0 ties with +0
    return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}

__device__ __forceinline__ uint32_t wave_inclusive_scan(uint32_t x, int lane) {
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const uint32_t y = __shfl_up(x, o, kWave);
        if (lane >= o) x += y;
    }
    return x;
}

// Exclusive prefix sum of v over the workgroup in thread order.
template <int NT>
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t *buf) {
    constexpr int NW = NT / kWave;
    const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x / kWave;
    const uint32_t incl = wave_inclusive_scan(v, lane);
    if (lane == kWave - 1) buf[w] = incl;
    __syncthreads();
    if (w == 0) {
        const uint32_t x = lane < NW ? buf[lane] : 0u;
        const uint32_t xi = wave_inclusive_scan(x, lane);
        if (lane < NW) buf[lane] = xi - x;
    }
    __syncthreads();
    const uint32_t r = buf[w] + incl - v;
    __syncthreads();
    return r;
}

// Where the keys come from: a unit's float64 energies, or (a unit of one
// token) the token's bf16 or fp32 activations.  For one token the energy of
// index j is x_j^2, which is exact in float64 and orders like |x_j|, whose
// IEEE bits (sign cleared) are already an unsigned order key: equal |x| tie
// exactly as equal squares do, +inf ranks above every finite value and every
// NaN is mapped to one key above +inf -- the order of the energy keys.
enum KeySrc { kEnergy = 0, kTokenBf16 = 1, kTokenF32 = 2 };

template <int SRC>
__device__ __forceinline__ uint64_t load_key(const void *row, int64_t j) {
    if constexpr (SRC == kEnergy) {
        return order_key(static_cast<const double *>(row)[j]);
    } else if constexpr (SRC == kTokenBf16) {
        uint32_t a = static_cast<const uint16_t *>(row)[j] & 0x7fffu;
        return a > 0x7f80u ? 0x7fc0u : a;
    } else {
        uint32_t a = static_cast<const uint32_t *>(row)[j] & 0x7fffffffu;
        return a > 0x7f800000u ? 0x7fc00000u : a;
    }
}

// NT threads; C keys per thread held in registers (REG) or re-read from
// memory (REG == false, chunk size `cpt` at run time).  Unit u's keys start
// at element u * ld of `src`.
template <int NT, int C, bool REG, int SRC>
__global__ __launch_bounds__(NT) void select_kernel(const void *__restrict__ src, int64_t ld,
                                                    int64_t K, int64_t k, int cpt,
                                                    int32_t *__restrict__ idx) {
    // lanes count into HR copies of the histogram (lane % HR), HR + 1 words
    // apart so that one digit's copies sit in different banks: the keys of a
    // unit often share a digit, and one copy would take most of a wave's
    // increments on one word
    constexpr int HR = 16, HS = 257;
    __shared__ uint32_t hcopy[HR * HS];
    __shared__ uint32_t hist[256];
    __shared__ uint32_t scan_buf[NT / kWave];
    __shared__ uint32_t s_digit, s_above, s_count;

    const int tid = threadIdx.x;
    constexpr int esize = SRC == kEnergy ? 8 : SRC == kTokenBf16 ? 2 : 4;
    const void *e = static_cast<const char *>(src) + static_cast<int64_t>(blockIdx.x) * ld * esize;
    int32_t *out = idx + static_cast<int64_t>(blockIdx.x) * k;
    const int chunk = REG ? C : cpt;
    const int64_t c0 = static_cast<int64_t>(tid) * chunk;

    if (k == K) {                       // everything is kept
        for (int64_t j = tid; j < K; j += NT) out[j] = static_cast<int32_t>(j);
        return;
    }

    uint64_t keys[REG ? C : 1];
    if constexpr (REG) {
#pragma unroll
        for (int c = 0; c < C; ++c) {
            const int64_t j = c0 + c;
            keys[c] = j < K ? load_key<SRC>(e, j) : 0ull;
        }
    }
    auto key_at = [&](int c) -> uint64_t {
        if constexpr (REG) return keys[c];
        else return load_key<SRC>(e, c0 + c);
    };
    const int n_own = static_cast<int>(max<int64_t>(0, min<int64_t>(chunk, K - c0)));

    // The leading bits shared by every key need no pass (energies of one
    // unit usually share sign and most of the exponent): take the
    // workgroup's smallest and largest key and start below their common
    // prefix, so the first pass already spreads the keys over its buckets.
    uint64_t kmin = ~0ull, kmax = 0;
    for (int c = 0; c < n_own; ++c) {
        const uint64_t u = key_at(c);
        kmin = u < kmin ? u : kmin;
        kmax = u > kmax ? u : kmax;
    }
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const uint64_t a = __shfl_xor(kmin, o, kWave), b = __shfl_xor(kmax, o, kWave);
        kmin = a < kmin ? a : kmin;
        kmax = b > kmax ? b : kmax;
    }
    __shared__ uint64_t s_min[NT / kWave], s_max[NT / kWave];
    if ((tid & (kWave - 1)) == 0) { s_min[tid / kWave] = kmin; s_max[tid / kWave] = kmax; }
    __syncthreads();
    kmin = s_min[0];
    kmax = s_max[0];
#pragma unroll
    for (int w = 1; w < NT / kWave; ++w) {
        kmin = s_min[w] < kmin ? s_min[w] : kmin;
        kmax = s_max[w] > kmax ? s_max[w] : kmax;
    }
    uint64_t prefix, mask;
    int top;                                        // highest bit not yet fixed
    if (kmin == kmax) {
        prefix = kmin; mask = ~0ull; top = -1;       // all keys equal: ties by index
    } else {
        top = 63 - __builtin_clzll(kmin ^ kmax);
        mask = top == 63 ? 0ull : (~0ull << (top + 1));
        prefix = kmax & mask;
    }
    uint32_t need = static_cast<uint32_t>(k);
    uint32_t *hmine = hcopy + (tid % HR) * HS;
    while (top >= 0) {
        // digit: bits top .. shift (up to 8 of them)
        const int shift = max(0, top - 7);
        const uint64_t dmask = (1ull << (top - shift + 1)) - 1;
        for (int i = tid; i < HR * HS; i += NT) hcopy[i] = 0;
        __syncthreads();
        if constexpr (REG) {
#pragma unroll
            for (int c = 0; c < C; ++c)
                if (c < n_own && (keys[c] & mask) == prefix)
                    atomicAdd(&hmine[(keys[c] >> shift) & dmask], 1u);
        } else {
            for (int c = 0; c < n_own; ++c) {
                const uint64_t u = key_at(c);
                if ((u & mask) == prefix) atomicAdd(&hmine[(u >> shift) & dmask], 1u);
            }
        }
        __syncthreads();
        for (int i = tid; i < 256; i += NT) {
            uint32_t t = 0;
#pragma unroll
            for (int r = 0; r < HR; ++r) t += hcopy[r * HS + i];
            hist[i] = t;
        }
        __syncthreads();
        if (tid < kWave) {
            // lane L holds digits 255-4L .. 252-4L (descending value order)
            uint32_t h[4], sum = 0;
#pragma unroll
            for (int q = 0; q < 4; ++q) { h[q] = hist[255 - 4 * tid - q]; sum += h[q]; }
            const uint32_t incl = wave_inclusive_scan(sum, tid);
            uint32_t run = incl - sum;
            if (run < need && need <= incl) {
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    if (run + h[q] >= need) {
                        s_digit = 255 - 4 * tid - q;
                        s_above = run;
                        s_count = h[q];
                        break;
                    }
                    run += h[q];
                }
            }
        }
        __syncthreads();
        need -= s_above;
        prefix |= static_cast<uint64_t>(s_digit) << shift;
        mask |= dmask << shift;
        top = shift - 1;
        if (s_count == need) break;      // the whole bucket is kept
    }

    // candidates share the prefix; keep the first `need` of them by index
    uint32_t n_cand = 0;
    for (int c = 0; c < n_own; ++c) n_cand += ((key_at(c) & mask) == prefix);
    uint32_t cand = block_exclusive_scan<NT>(n_cand, scan_buf);
    uint32_t n_sel = 0;
    {
        uint32_t cc = cand;
        for (int c = 0; c < n_own; ++c) {
            const uint64_t p = key_at(c) & mask;
            if (p > prefix) ++n_sel;
            else if (p == prefix) { n_sel += (cc < need); ++cc; }
        }
    }
    uint32_t pos = block_exclusive_scan<NT>(n_sel, scan_buf);
    for (int c = 0; c < n_own; ++c) {
        const uint64_t p = key_at(c) & mask;
        bool keep = p > prefix;
        if (p == prefix) { keep = cand < need; ++cand; }
        if (keep) out[pos++] = static_cast<int32_t>(c0 + c);
    }
}

// One bf16 token per workgroup (a decode step), K <= 32 * 1024 (at most
// 32768 keys, so both 16-bit halves of the packed scan below hold): the keys are
// the 15 magnitude bits, so the k-th largest key is found in at most two
// histogram passes (bits 14..7, then 6..0), each of the NT threads owning C
// consecutive keys loaded as 16-byte vectors.  The kept set is then
// written in ascending order after one scan of a packed pair per thread
// (keys above the threshold | ties with it << 16): a kept key's slot is the
// number of kept keys before it, i.e. keys above before it plus
// min(ties before it, ties kept).
template <int NT, int C>
__device__ __forceinline__ void select_token16(const uint16_t *__restrict__ x, int K, int k,
                                               int32_t *__restrict__ out) {
    static_assert(C % 8 == 0 && C <= 32 && NT >= 256 && NT <= 1024, "chunk");
    // The keys of a token bunch up in a few digits (one per binary exponent),
    // so one histogram would take most of a wave's 64 increments on one
    // word.  Lanes count into HR copies (lane % HR), HR + 1 words apart so
    // that one digit's copies sit in different banks, and the copies are
    // summed before the scan.
    constexpr int HR = 16, HS = 257;
    __shared__ uint32_t hcopy[HR * HS];
    __shared__ uint32_t hist[256];
    __shared__ uint32_t scan_buf[NT / kWave];
    __shared__ int s_thr, s_need;
    const int tid = threadIdx.x, lane = tid & (kWave - 1);
    if (k == K) {                       // everything is kept
        for (int j = tid; j < K; j += NT) out[j] = j;
        return;
    }
    const int c0 = tid * C;
    // keys past K are marked with bit 15 and never counted
    uint32_t key[C];
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t *>(x), 0, static_cast<uint32_t>(K) * 2u, 0x00020000);
#pragma unroll
    for (int q = 0; q < C / 8; ++q) {
        const auto v = __builtin_amdgcn_raw_buffer_load_b128(xr, static_cast<uint32_t>(c0 + 8 * q) * 2u, 0, 0);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const uint32_t h = (v[e / 2] >> (16 * (e % 2))) & 0x7fffu;
            key[8 * q + e] = c0 + 8 * q + e < K ? (h > 0x7f80u ? 0x7fc0u : h) : 0x8000u;
        }
    }
    // pass 1 over bits 14..7, pass 2 over bits 6..0 of the keys in the chosen bucket
    int need = k, thr = -1, take_ties = 0;
    int prefix = -1;                    // pass-1 digit, once chosen
    uint32_t *hmine = hcopy + (lane % HR) * HS;
#pragma unroll
    for (int pass = 0; pass < 2; ++pass) {
        for (int j = tid; j < HR * HS; j += NT) hcopy[j] = 0;
        __syncthreads();
#pragma unroll
        for (int c = 0; c < C; ++c) {
            const uint32_t u = key[c];
            if (u & 0x8000u) continue;
            if (pass == 0) atomicAdd(&hmine[u >> 7], 1u);
            else if (static_cast<int>(u >> 7) == prefix) atomicAdd(&hmine[u & 0x7fu], 1u);
        }
        __syncthreads();
        if (tid < 256) {
            uint32_t t = 0;
#pragma unroll
            for (int r = 0; r < HR; ++r) t += hcopy[r * HS + tid];
            hist[tid] = t;
        }
        __syncthreads();
        if (tid < kWave) {
            // lane L holds digits 255-4L .. 252-4L (descending value order)
            uint32_t h[4], sum = 0;
#pragma unroll
            for (int q = 0; q < 4; ++q) { h[q] = hist[255 - 4 * lane - q]; sum += h[q]; }
            const uint32_t incl = wave_inclusive_scan(sum, lane);
            uint32_t run = incl - sum;
            const uint32_t nd = static_cast<uint32_t>(need);
            if (run < nd && nd <= incl) {
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    if (run + h[q] >= nd) {
                        s_thr = 255 - 4 * lane - q;
                        s_need = static_cast<int>(nd - run);   // keys of this bucket to keep
                        hist[0] = h[q];                        // its size (read after the barrier)
                        break;
                    }
                    run += h[q];
                }
            }
        }
        __syncthreads();
        const int d = s_thr, nb = s_need, size = static_cast<int>(hist[0]);
        __syncthreads();                // hist is rewritten by the next pass
        if (pass == 0) {
            if (size == nb) { thr = (d << 7) - 1; take_ties = 0; break; }   // the whole bucket
            prefix = d;
            need = nb;
        } else {
            thr = (prefix << 7) | d;    // the k-th largest key; keep nb of its ties
            take_ties = nb;
        }
    }
    // compaction: keys above thr, then the first take_ties keys equal to thr
    uint32_t above = 0, ties = 0;
#pragma unroll
    for (int c = 0; c < C; ++c) {
        const int u = static_cast<int>(key[c]);
        above += u < 0x8000 && u > thr;
        ties += u == thr;
    }
    const uint32_t pre = block_exclusive_scan<NT>(above | (ties << 16), scan_buf);
    int sa = static_cast<int>(pre & 0xffffu), st = static_cast<int>(pre >> 16);
#pragma unroll
    for (int c = 0; c < C; ++c) {
        const int u = static_cast<int>(key[c]);
        if (u < 0x8000 && u > thr) {
            out[sa + min(st, take_ties)] = c0 + c;
            ++sa;
        } else if (u == thr) {
            if (st < take_ties) out[sa + st] = c0 + c;
            ++st;
        }
    }
}

template <int NT, int C>
__global__ __launch_bounds__(NT) void select_token16_kernel(const uint16_t *__restrict__ X,
                                                            int64_t ldx, int K, int k,
                                                            int32_t *__restrict__ idx) {
    select_token16<NT, C>(X + static_cast<int64_t>(blockIdx.x) * ldx, K, k,
                          idx + static_cast<int64_t>(blockIdx.x) * k);
}

// the token selection of several groups in one launch: workgroup (b, g)
// takes unit b of group g
__global__ __launch_bounds__(1024) void select_token16_grouped_kernel(GemvGroups G) {
    const GemvGroup &q = G.g[blockIdx.y];
    if (q.K > kToken16MaxK) return;              // selected by a launch of its own
    const uint16_t *x = q.X + static_cast<int64_t>(blockIdx.x) * q.ldx;
    int32_t *out = q.idx_out + static_cast<int64_t>(blockIdx.x) * q.k;
    if (q.K <= 16 * 1024) select_token16<1024, 16>(x, q.K, q.k, out);   // uniform per workgroup
    else select_token16<1024, 32>(x, q.K, q.k, out);
}

template <int NT, int C>
hipError_t launch_token16(const void *X, int64_t ldx, int64_t B, int64_t K, int64_t k, int32_t *idx,
                          hipStream_t stream) {
    hipLaunchKernelGGL((select_token16_kernel<NT, C>), dim3(static_cast<unsigned>(B)), dim3(NT), 0, stream,
                       static_cast<const uint16_t *>(X), ldx, static_cast<int>(K), static_cast<int>(k), idx);
    return hipGetLastError();
}

template <int NT, int C, bool REG, int SRC>
hipError_t launch(const void *src, int64_t ld, int64_t B, int64_t K, int64_t k, int cpt,
                  int32_t *idx, hipStream_t stream) {
    hipLaunchKernelGGL((select_kernel<NT, C, REG, SRC>), dim3(static_cast<unsigned>(B)), dim3(NT), 0,
                       stream, src, ld, K, k, cpt, idx);
    return hipGetLastError();
}

template <int SRC>
hipError_t launch_src(const void *src, int64_t ld, int64_t B, int64_t K, int64_t k, int32_t *idx,
                      hipStream_t stream) {
    if (K <= 256) return launch<256, 1, true, SRC>(src, ld, B, K, k, 1, idx, stream);
    if (K <= 512) return launch<256, 2, true, SRC>(src, ld, B, K, k, 2, idx, stream);
    if (K <= 1024) return launch<256, 4, true, SRC>(src, ld, B, K, k, 4, idx, stream);
    if (K <= 2048) return launch<256, 8, true, SRC>(src, ld, B, K, k, 8, idx, stream);
    if (K <= 4096) return launch<1024, 4, true, SRC>(src, ld, B, K, k, 4, idx, stream);
    if (K <= 8192) return launch<1024, 8, true, SRC>(src, ld, B, K, k, 8, idx, stream);
    if (K <= 16384) return launch<1024, 16, true, SRC>(src, ld, B, K, k, 16, idx, stream);
    if (K <= 32768) return launch<1024, 32, true, SRC>(src, ld, B, K, k, 32, idx, stream);
    const int cpt = static_cast<int>((K + 1023) / 1024);
    return launch<1024, 1, false, SRC>(src, ld, B, K, k, cpt, idx, stream);
}

// bad[b] = 0 when unit b's list idx[b*k .. b*k+k) is strictly ascending with
// every value in [0, K), else 1 + the first position t that breaks it
// (idx[t] out of range, or idx[t] <= idx[t-1]).  Integer work: the first
// position is an integer minimum over the threads, order-free.
__global__ __launch_bounds__(256) void check_indices_kernel(const int32_t *__restrict__ idx,
                                                            int64_t k, int32_t K,
                                                            int32_t *__restrict__ bad) {
    __shared__ int first;
    const int32_t *I = idx + static_cast<int64_t>(blockIdx.x) * k;
    if (threadIdx.x == 0) first = 0x7fffffff;
    __syncthreads();
    for (int64_t t = threadIdx.x; t < k; t += 256) {
        const int32_t v = I[t];
        if (v < 0 || v >= K || (t > 0 && I[t - 1] >= v)) {
            atomicMin(&first, static_cast<int>(t));      // t grows along a thread's loop
            break;
        }
    }
    __syncthreads();
    if (threadIdx.x == 0) bad[blockIdx.x] = first == 0x7fffffff ? 0 : first + 1;
}

}  // namespace

hipError_t launch_check_indices(const int32_t *idx, int64_t B, int64_t k, int64_t K, int32_t *bad,
                                hipStream_t stream) {
    hipLaunchKernelGGL(check_indices_kernel, dim3(static_cast<unsigned>(B)), dim3(256), 0, stream,
                       idx, k, static_cast<int32_t>(K), bad);
    return hipGetLastError();
}

hipError_t launch_select(const double *energy, int64_t B, int64_t K, int64_t k,
                         int32_t *idx, hipStream_t stream) {
    return launch_src<kEnergy>(energy, K, B, K, k, idx, stream);
}

hipError_t launch_select_tokens_grouped(const GemvGroups &G, int64_t B, hipStream_t stream) {
    hipLaunchKernelGGL(select_token16_grouped_kernel, dim3(static_cast<unsigned>(B), static_cast<unsigned>(G.n)),
                       dim3(1024), 0, stream, G);
    hipError_t e = hipGetLastError();
    // groups too wide for the one-pass token kernel: the generic selection
    for (int i = 0; i < G.n && e == hipSuccess; ++i) {
        const GemvGroup &q = G.g[i];
        if (q.K > kToken16MaxK)
            e = launch_select_tokens(q.X, true, B, q.K, q.ldx, q.k, q.idx_out, stream);
    }
    return e;
}

hipError_t launch_select_tokens(const void *X, bool bf16, int64_t B, int64_t K, int64_t ldx,
                                int64_t k, int32_t *idx, hipStream_t stream) {
    if (bf16 && K <= kToken16MaxK && reinterpret_cast<uintptr_t>(X) % 16 == 0 && ldx % 8 == 0) {
        if (K <= 8 * 256) return launch_token16<256, 8>(X, ldx, B, K, k, idx, stream);
        if (K <= 16 * 256) return launch_token16<256, 16>(X, ldx, B, K, k, idx, stream);
        if (K <= 16 * 512) return launch_token16<512, 16>(X, ldx, B, K, k, idx, stream);
        if (K <= 16 * 1024) return launch_token16<1024, 16>(X, ldx, B, K, k, idx, stream);
        return launch_token16<1024, 32>(X, ldx, B, K, k, idx, stream);
    }
    return bf16 ? launch_src<kTokenBf16>(X, ldx, B, K, k, idx, stream)
                : launch_src<kTokenF32>(X, ldx, B, K, k, idx, stream);
}

}  // namespace rmm
