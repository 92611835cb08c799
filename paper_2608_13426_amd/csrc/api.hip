// C-ABI of librmm: host-side validation, the k = ceil(r*K) rule, workspace
// layout and dispatch to the gfx950 kernels.  Every check happens before
// the first HIP call, so invalid calls never touch the device.
#include <cmath>
#include <cstdint>

#include "../../include/rmm.h"
#include "kernels.h"
#include "gemv_shared.h"

namespace {

constexpr int64_t kInt32Max = 2147483647;
constexpr int64_t kGridYZMax = 65535;

inline size_t align256(size_t n) { return (n + 255) & ~static_cast<size_t>(255); }

inline bool valid_dtype(rmm_dtype_t dt) { return dt == RMM_F32 || dt == RMM_BF16; }

inline rmm_status_t from_hip(hipError_t e) { return e == hipSuccess ? RMM_OK : RMM_ERR_HIP; }

rmm_status_t check_score(const void *X, rmm_dtype_t dt, int64_t B, int64_t M, int64_t K,
                         int64_t ldx, const double *energy) {
    if (!X || !energy) return RMM_ERR_INVALID_ARGUMENT;
    if (!valid_dtype(dt)) return RMM_ERR_INVALID_ARGUMENT;
    if (B < 1 || M < 1 || K < 1 || ldx < K) return RMM_ERR_INVALID_ARGUMENT;
    if (K > kInt32Max) return RMM_ERR_INVALID_ARGUMENT;
    if (B > kGridYZMax) return RMM_ERR_UNSUPPORTED;
    return RMM_OK;
}

// Checks shared by rmm_reduced_gemm and rmm_linear (whose index list lives
// in the workspace or idx_out, so it has no idx pointer to check here).
rmm_status_t check_gemm_shapes(const void *X, const void *W, rmm_dtype_t dt, int64_t B,
                               int64_t M, int64_t N, int64_t K, int64_t k, int64_t ldx,
                               int64_t ldw, const void *Y, int64_t ldy) {
    if (!X || !W || !Y) return RMM_ERR_INVALID_ARGUMENT;
    if (!valid_dtype(dt)) return RMM_ERR_INVALID_ARGUMENT;
    if (B < 1 || M < 1 || N < 1 || K < 1) return RMM_ERR_INVALID_ARGUMENT;
    if (k < 1 || k > K) return RMM_ERR_INVALID_ARGUMENT;
    if (ldx < K || ldw < N || ldy < N) return RMM_ERR_INVALID_ARGUMENT;
    if (K > kInt32Max || M > kInt32Max || N > kInt32Max) return RMM_ERR_INVALID_ARGUMENT;
    if (B > kGridYZMax || M > kGridYZMax * 64) return RMM_ERR_UNSUPPORTED;
    return RMM_OK;
}

inline bool aligned16(const void *p) { return reinterpret_cast<uintptr_t>(p) % 16 == 0; }

// The K-major GEMM reads 16-byte vectors through buffer descriptors whose
// byte offsets must stay below 2^31.
bool kmajor_ok(const void *Xt, const void *W, int64_t B, int64_t M, int64_t K, int64_t ldxt,
               int64_t ldw) {
    if (!aligned16(Xt) || !aligned16(W) || ldxt % 8 || ldw % 8) return false;
    const int64_t lim = int64_t(1) << 31;
    if (K * ldxt * 2 + ldxt * 2 >= lim || K * ldw * 2 + ldw * 2 >= lim) return false;
    return B <= kGridYZMax && M <= kInt32Max;
}

// K-major copy of the activations held in rmm_linear's workspace
inline int64_t xt_ld(int64_t M) { return (M + 7) / 8 * 8; }
inline size_t xt_bytes(int64_t B, int64_t M, int64_t K) {
    return static_cast<size_t>(B * K * xt_ld(M)) * 2;
}

}  // namespace

extern "C" {

int64_t rmm_retained_count(double r, int64_t K) {
    if (K < 1 || K > kInt32Max) return -1;
    if (!(r > 0.0 && r <= 1.0)) return -1;     // also rejects NaN
    const double p = r * static_cast<double>(K);
    const double nearest = std::nearbyint(p);
    int64_t k;
    if (std::fabs(p - nearest) <= 1e-9 * static_cast<double>(K))
        k = static_cast<int64_t>(nearest);
    else
        k = static_cast<int64_t>(std::ceil(p));
    if (k < 1) k = 1;
    if (k > K) k = K;
    return k;
}

size_t rmm_workspace_size(rmm_op_t op, int64_t B, int64_t M, int64_t K, int64_t k) {
    if (B < 1 || K < 1) return 0;
    switch (op) {
    case RMM_OP_SCORE:
        return M < 1 ? 0 : rmm::score_workspace_bytes(B, M, K);
    case RMM_OP_SELECT:
        return 0;
    case RMM_OP_LINEAR:
    case RMM_OP_PV:
        if (M < 1 || k < 1 || k > K) return 0;
        return align256(rmm::score_workspace_bytes(B, M, K)) +
               align256(static_cast<size_t>(B * K) * sizeof(double)) +
               align256(static_cast<size_t>(B * k) * sizeof(int32_t)) + align256(xt_bytes(B, M, K));
    case RMM_OP_ATTENTION:
        if (M < 1 || k < 1 || k > K) return 0;
        return align256(rmm::attn_workspace_bytes(B, M, k));
    }
    return 0;
}

rmm_status_t rmm_score(const void *X, rmm_dtype_t dtype, int64_t B, int64_t M, int64_t K,
                       int64_t ldx, double *energy, void *workspace, size_t workspace_bytes,
                       hipStream_t stream) {
    rmm_status_t st = check_score(X, dtype, B, M, K, ldx, energy);
    if (st != RMM_OK) return st;
    const size_t need = rmm::score_workspace_bytes(B, M, K);
    if (need > 0) {
        if (!workspace || workspace_bytes < need) return RMM_ERR_WORKSPACE_TOO_SMALL;
        if (reinterpret_cast<uintptr_t>(workspace) % 8) return RMM_ERR_INVALID_ARGUMENT;
    }
    return from_hip(rmm::launch_score(X, dtype == RMM_BF16, B, M, K, ldx, energy,
                                      static_cast<double *>(workspace), nullptr, 0, stream));
}

rmm_status_t rmm_score_kmajor(const void *X, int64_t B, int64_t M, int64_t K, int64_t ldx,
                              double *energy, void *Xt, int64_t ldxt, void *workspace,
                              size_t workspace_bytes, hipStream_t stream) {
    rmm_status_t st = check_score(X, RMM_BF16, B, M, K, ldx, energy);
    if (st != RMM_OK) return st;
    if (!Xt || ldxt < M) return RMM_ERR_INVALID_ARGUMENT;
    if (!aligned16(X) || ldx % 8 || !aligned16(Xt) || ldxt % 8) return RMM_ERR_UNSUPPORTED;
    const size_t need = rmm::score_workspace_bytes(B, M, K);
    if (need > 0) {
        if (!workspace || workspace_bytes < need) return RMM_ERR_WORKSPACE_TOO_SMALL;
        if (reinterpret_cast<uintptr_t>(workspace) % 8) return RMM_ERR_INVALID_ARGUMENT;
    }
    return from_hip(rmm::launch_score(X, true, B, M, K, ldx, energy, static_cast<double *>(workspace),
                                      static_cast<uint16_t *>(Xt), ldxt, stream));
}

size_t rmm_rmsnorm_kmajor_workspace_size(int64_t B, int64_t M, int64_t K) {
    if (B < 1 || M < 1 || K < 1) return 0;
    return align256(rmm::rmsnorm_workspace_bytes(B, M, K));
}

rmm_status_t rmm_rmsnorm_kmajor(const void *X, const void *gamma, float eps, int64_t B, int64_t M,
                                int64_t K, int64_t ldx, void *Xt, int64_t ldxt, double *energy,
                                void *workspace, size_t workspace_bytes, hipStream_t stream) {
    if (!X || !gamma || !Xt || !energy) return RMM_ERR_INVALID_ARGUMENT;
    if (B < 1 || M < 1 || K < 1 || ldx < K || ldxt < M) return RMM_ERR_INVALID_ARGUMENT;
    if (!(eps >= 0.f) || std::isinf(eps)) return RMM_ERR_INVALID_ARGUMENT;   // also NaN
    if (M > kInt32Max) return RMM_ERR_INVALID_ARGUMENT;
    if (K % 8 || K > kInt32Max || B > kGridYZMax) return RMM_ERR_UNSUPPORTED;
    // the two-pass tile kernel addresses one row split with 32-bit byte offsets
    if (!rmm::rmsnorm_single_pass(K, ldx) &&
        rmm::score_rows_per_split(B, M, K) * ldx * 2 >= (int64_t(1) << 31))
        return RMM_ERR_UNSUPPORTED;
    if (!aligned16(X) || !aligned16(gamma) || !aligned16(Xt) || ldx % 8 || ldxt % 8 ||
        reinterpret_cast<uintptr_t>(energy) % 8)
        return RMM_ERR_UNSUPPORTED;
    const size_t need = rmm_rmsnorm_kmajor_workspace_size(B, M, K);
    if (!workspace || workspace_bytes < need) return RMM_ERR_WORKSPACE_TOO_SMALL;
    if (reinterpret_cast<uintptr_t>(workspace) % 256) return RMM_ERR_INVALID_ARGUMENT;
    return from_hip(rmm::launch_rmsnorm_kmajor(
        static_cast<const uint16_t *>(X), static_cast<const uint16_t *>(gamma), eps, B, M, K, ldx,
        static_cast<uint16_t *>(Xt), ldxt, energy, workspace, stream));
}

rmm_status_t rmm_select(const double *energy, int64_t B, int64_t K, int64_t k, int32_t *idx,
                        hipStream_t stream) {
    if (!energy || !idx) return RMM_ERR_INVALID_ARGUMENT;
    if (B < 1 || K < 1 || k < 1 || k > K || K > kInt32Max) return RMM_ERR_INVALID_ARGUMENT;
    if (B > kInt32Max) return RMM_ERR_UNSUPPORTED;
    return from_hip(rmm::launch_select(energy, B, K, k, idx, stream));
}

rmm_status_t rmm_check_indices(const int32_t *idx, int64_t B, int64_t k, int64_t K, int32_t *bad,
                               hipStream_t stream) {
    if (!idx || !bad) return RMM_ERR_INVALID_ARGUMENT;
    if (B < 1 || K < 1 || k < 1 || k > K || K > kInt32Max) return RMM_ERR_INVALID_ARGUMENT;
    if (B > kInt32Max) return RMM_ERR_UNSUPPORTED;
    return from_hip(rmm::launch_check_indices(idx, B, k, K, bad, stream));
}

rmm_status_t rmm_reduced_gemm(const void *X, const void *W, const int32_t *idx, rmm_dtype_t dtype,
                              int64_t B, int64_t M, int64_t N, int64_t K, int64_t k, int64_t ldx,
                              int64_t ldw, void *Y, int64_t ldy, hipStream_t stream) {
    if (!idx) return RMM_ERR_INVALID_ARGUMENT;
    rmm_status_t st = check_gemm_shapes(X, W, dtype, B, M, N, K, k, ldx, ldw, Y, ldy);
    if (st != RMM_OK) return st;
    if (dtype == RMM_BF16)
        return from_hip(rmm::launch_gemm_bf16(
            static_cast<const uint16_t *>(X), static_cast<const uint16_t *>(W), idx, B, M, N, K, k,
            ldx, ldw, static_cast<uint16_t *>(Y), ldy, stream));
    return from_hip(rmm::launch_gemm_f32(static_cast<const float *>(X),
                                         static_cast<const float *>(W), idx, B, M, N, K, k, ldx,
                                         ldw, static_cast<float *>(Y), ldy, stream));
}

rmm_status_t rmm_select_tokens(const void *X, rmm_dtype_t dtype, int64_t B, int64_t K,
                               int64_t ldx, int64_t k, int32_t *idx, hipStream_t stream) {
    if (!X || !idx) return RMM_ERR_INVALID_ARGUMENT;
    if (!valid_dtype(dtype)) return RMM_ERR_INVALID_ARGUMENT;
    if (B < 1 || K < 1 || k < 1 || k > K || ldx < K) return RMM_ERR_INVALID_ARGUMENT;
    if (K > kInt32Max) return RMM_ERR_INVALID_ARGUMENT;
    if (B > kInt32Max) return RMM_ERR_UNSUPPORTED;
    return from_hip(rmm::launch_select_tokens(X, dtype == RMM_BF16, B, K, ldx, k, idx, stream));
}

size_t rmm_gemv_workspace_size(int64_t B, int64_t M, int64_t N, int64_t k) {
    if (B < 1 || M < 1 || M > 8 || N < 1 || k < 1) return 0;
    const size_t b = rmm::gemv_workspace_bytes(B, M, N, k);
    return b == 0 ? 0 : align256(b);
}

rmm_status_t rmm_reduced_gemv(const void *X, const void *W, const int32_t *idx, rmm_dtype_t dtype,
                              int64_t B, int64_t M, int64_t N, int64_t K, int64_t k, int64_t ldx,
                              int64_t ldw, void *Y, int64_t ldy, void *workspace,
                              size_t workspace_bytes, hipStream_t stream) {
    if (!idx) return RMM_ERR_INVALID_ARGUMENT;
    rmm_status_t st = check_gemm_shapes(X, W, dtype, B, M, N, K, k, ldx, ldw, Y, ldy);
    if (st != RMM_OK) return st;
    if (dtype != RMM_BF16 || M > 8) return RMM_ERR_UNSUPPORTED;
    // 32-bit byte offsets into W (the kernel reads it through one descriptor)
    if (K * ldw * 2 >= (int64_t(1) << 31)) return RMM_ERR_UNSUPPORTED;
    const size_t need = rmm::gemv_workspace_bytes(B, M, N, k);
    if (need > 0) {
        if (!workspace || workspace_bytes < need) return RMM_ERR_WORKSPACE_TOO_SMALL;
        if (reinterpret_cast<uintptr_t>(workspace) % 16) return RMM_ERR_INVALID_ARGUMENT;
    }
    return from_hip(rmm::launch_gemv_bf16(static_cast<const uint16_t *>(X),
                                          static_cast<const uint16_t *>(W), idx, B, M, N, K, k, ldx,
                                          ldw, static_cast<uint16_t *>(Y), ldy, workspace, stream));
}

rmm_status_t rmm_reduced_gemm_kmajor(const void *Xt, const void *W, const int32_t *idx, int64_t B,
                                     int64_t M, int64_t N, int64_t K, int64_t k, int64_t ldxt,
                                     int64_t ldw, void *Y, int64_t ldy, hipStream_t stream) {
    if (!Xt || !W || !idx || !Y) return RMM_ERR_INVALID_ARGUMENT;
    if (B < 1 || M < 1 || N < 1 || K < 1 || k < 1 || k > K) return RMM_ERR_INVALID_ARGUMENT;
    if (ldxt < M || ldw < N || ldy < N) return RMM_ERR_INVALID_ARGUMENT;
    if (K > kInt32Max || M > kInt32Max || N > kInt32Max) return RMM_ERR_INVALID_ARGUMENT;
    if (!kmajor_ok(Xt, W, B, M, K, ldxt, ldw)) return RMM_ERR_UNSUPPORTED;
    return from_hip(rmm::launch_gemm_kmajor_bf16(static_cast<const uint16_t *>(Xt),
                                                 static_cast<const uint16_t *>(W), idx, B, M, N, K, k,
                                                 ldxt, ldw, static_cast<uint16_t *>(Y), ldy, stream));
}

size_t rmm_gemm_swiglu_workspace_size(int64_t B, int64_t M, int64_t F) {
    if (B < 1 || M < 1 || F < 1) return 0;
    return align256(static_cast<size_t>(B * ((M + 255) / 256) * F) * sizeof(double));
}

rmm_status_t rmm_reduced_gemm_swiglu_kmajor(const void *Xt, const void *Wgu, const int32_t *idx,
                                            int64_t B, int64_t M, int64_t F, int64_t K, int64_t k,
                                            int64_t ldxt, int64_t ldw, void *Ht, int64_t ldht,
                                            double *energy, void *workspace,
                                            size_t workspace_bytes, hipStream_t stream) {
    if (!Xt || !Wgu || !idx || !Ht || !energy) return RMM_ERR_INVALID_ARGUMENT;
    if (B < 1 || M < 1 || F < 1 || K < 1 || k < 1 || k > K) return RMM_ERR_INVALID_ARGUMENT;
    if (ldxt < M || ldw < 2 * F || ldht < M) return RMM_ERR_INVALID_ARGUMENT;
    if (K > kInt32Max || M > kInt32Max || 2 * F > kInt32Max) return RMM_ERR_INVALID_ARGUMENT;
    if (!kmajor_ok(Xt, Wgu, B, M, K, ldxt, ldw)) return RMM_ERR_UNSUPPORTED;
    if (F % 128 || M % 8 || ldht % 8 || !aligned16(Ht) || reinterpret_cast<uintptr_t>(energy) % 8)
        return RMM_ERR_UNSUPPORTED;
    if ((M + 255) / 256 * (F / 128) > kInt32Max) return RMM_ERR_UNSUPPORTED;
    const size_t need = rmm_gemm_swiglu_workspace_size(B, M, F);
    if (!workspace || workspace_bytes < need) return RMM_ERR_WORKSPACE_TOO_SMALL;
    if (reinterpret_cast<uintptr_t>(workspace) % 8) return RMM_ERR_INVALID_ARGUMENT;
    return from_hip(rmm::launch_gemm_swiglu_kmajor_bf16(
        static_cast<const uint16_t *>(Xt), static_cast<const uint16_t *>(Wgu), idx, B, M, F, K, k,
        ldxt, ldw, static_cast<uint16_t *>(Ht), ldht, energy, static_cast<double *>(workspace),
        stream));
}

rmm_status_t rmm_reduced_qk(const void *Q, const void *Kc, const int32_t *idx, rmm_dtype_t dtype,
                            int64_t batch, int64_t H, int64_t Hkv, int64_t Lq, int64_t Lk,
                            int64_t D, int64_t k, float scale, int causal, void *S,
                            hipStream_t stream) {
    if (!Q || !Kc || !idx || !S) return RMM_ERR_INVALID_ARGUMENT;
    if (!valid_dtype(dtype)) return RMM_ERR_INVALID_ARGUMENT;
    if (batch < 1 || H < 1 || Hkv < 1 || Lq < 1 || Lk < 1 || D < 1) return RMM_ERR_INVALID_ARGUMENT;
    if (H % Hkv != 0) return RMM_ERR_INVALID_ARGUMENT;
    if (k < 1 || k > D) return RMM_ERR_INVALID_ARGUMENT;
    if (Lq > kInt32Max || Lk > kInt32Max) return RMM_ERR_INVALID_ARGUMENT;
    if (D > 256) return RMM_ERR_UNSUPPORTED;
    if (batch * H > kGridYZMax || Lq > kGridYZMax * 64) return RMM_ERR_UNSUPPORTED;
    if (dtype == RMM_BF16)
        return from_hip(rmm::launch_qk_bf16(static_cast<const uint16_t *>(Q),
                                            static_cast<const uint16_t *>(Kc), idx, batch, H, Hkv,
                                            Lq, Lk, D, k, scale, causal != 0,
                                            static_cast<uint16_t *>(S), stream));
    return from_hip(rmm::launch_qk_f32(static_cast<const float *>(Q), static_cast<const float *>(Kc),
                                       idx, batch, H, Hkv, Lq, Lk, D, k, scale, causal != 0,
                                       static_cast<float *>(S), stream));
}

rmm_status_t rmm_reduced_qk_rowstats(const void *Q, const void *Kc, const int32_t *idx, int64_t batch,
                                     int64_t H, int64_t Hkv, int64_t Lq, int64_t Lk, int64_t D,
                                     int64_t k, float scale, int causal, void *S, float *row_max,
                                     float *row_rinv, hipStream_t stream) {
    if (!Q || !Kc || !idx || !S || !row_max || !row_rinv) return RMM_ERR_INVALID_ARGUMENT;
    if (batch < 1 || H < 1 || Hkv < 1 || Lq < 1 || Lk < 1 || D < 1) return RMM_ERR_INVALID_ARGUMENT;
    if (H % Hkv != 0) return RMM_ERR_INVALID_ARGUMENT;
    if (k < 1 || k > D) return RMM_ERR_INVALID_ARGUMENT;
    if (Lq > kInt32Max || Lk > kInt32Max) return RMM_ERR_INVALID_ARGUMENT;
    if (batch * H > kGridYZMax || Lq > kGridYZMax * 64) return RMM_ERR_UNSUPPORTED;
    if (!rmm::qk_rows_ok(Lk, D, S) || reinterpret_cast<uintptr_t>(row_max) % 4 ||
        reinterpret_cast<uintptr_t>(row_rinv) % 4)
        return RMM_ERR_UNSUPPORTED;
    const hipError_t e = rmm::launch_qk_rowstats_bf16(
        static_cast<const uint16_t *>(Q), static_cast<const uint16_t *>(Kc), idx, batch, H, Hkv, Lq, Lk,
        D, k, scale, causal != 0, static_cast<uint16_t *>(S), row_max, row_rinv, stream);
    return e == hipErrorNotSupported ? RMM_ERR_UNSUPPORTED : from_hip(e);
}

rmm_status_t rmm_reduced_attention(const void *Q, const void *Kc, const void *V,
                                   const int32_t *idx, rmm_dtype_t dtype, int64_t batch,
                                   int64_t H, int64_t Hkv, int64_t Lq, int64_t Lk, int64_t D,
                                   int64_t k, float scale, int causal, void *O,
                                   void *workspace, size_t workspace_bytes, hipStream_t stream) {
    if (!Q || !Kc || !V || !idx || !O) return RMM_ERR_INVALID_ARGUMENT;
    if (!valid_dtype(dtype)) return RMM_ERR_INVALID_ARGUMENT;
    if (batch < 1 || H < 1 || Hkv < 1 || Lq < 1 || Lk < 1 || D < 1) return RMM_ERR_INVALID_ARGUMENT;
    if (H % Hkv != 0) return RMM_ERR_INVALID_ARGUMENT;
    if (k < 1 || k > D) return RMM_ERR_INVALID_ARGUMENT;
    if (Lq > kInt32Max || Lk > kInt32Max) return RMM_ERR_INVALID_ARGUMENT;
    if (dtype != RMM_BF16 || D != 128) return RMM_ERR_UNSUPPORTED;
    if (!aligned16(Q) || !aligned16(Kc) || !aligned16(V) || !aligned16(O)) return RMM_ERR_UNSUPPORTED;
    if (batch * H > kGridYZMax || (Lq + 255) / 256 * batch * H > kInt32Max) return RMM_ERR_UNSUPPORTED;
    if (!workspace || workspace_bytes < rmm::attn_workspace_bytes(batch * H, Lk, k))
        return RMM_ERR_WORKSPACE_TOO_SMALL;
    if (!aligned16(workspace)) return RMM_ERR_INVALID_ARGUMENT;
    return from_hip(rmm::launch_attn_bf16(
        static_cast<const uint16_t *>(Q), static_cast<const uint16_t *>(Kc),
        static_cast<const uint16_t *>(V), idx, batch, H, Hkv, Lq, Lk, k, scale, causal != 0,
        static_cast<uint16_t *>(O), workspace, stream));
}

size_t rmm_attention_kmajor_workspace_size(int64_t batch, int64_t H, int64_t Lq, int64_t Lk,
                                            int64_t D, int64_t k) {
    if (batch < 1 || H < 1 || Lq < 1 || Lk < 1 || D < 1 || k < 1 || k > D) return 0;
    return align256(rmm::attn_workspace_bytes(batch * H, Lk, k)) +
           align256(static_cast<size_t>(batch * rmm::attn_query_tiles(Lq) * H * D) * sizeof(double));
}

rmm_status_t rmm_reduced_attention_kmajor(const void *Q, const void *Kc, const void *V,
                                          const int32_t *idx, rmm_dtype_t dtype, int64_t batch,
                                          int64_t H, int64_t Hkv, int64_t Lq, int64_t Lk,
                                          int64_t D, int64_t k, float scale, int causal, void *Ot,
                                          int64_t ldot, double *energy, void *workspace,
                                          size_t workspace_bytes, hipStream_t stream) {
    if (!Q || !Kc || !V || !idx || !Ot || !energy) return RMM_ERR_INVALID_ARGUMENT;
    if (!valid_dtype(dtype)) return RMM_ERR_INVALID_ARGUMENT;
    if (batch < 1 || H < 1 || Hkv < 1 || Lq < 1 || Lk < 1 || D < 1) return RMM_ERR_INVALID_ARGUMENT;
    if (H % Hkv != 0) return RMM_ERR_INVALID_ARGUMENT;
    if (k < 1 || k > D) return RMM_ERR_INVALID_ARGUMENT;
    if (Lq > kInt32Max || Lk > kInt32Max || ldot < Lq) return RMM_ERR_INVALID_ARGUMENT;
    if (dtype != RMM_BF16 || D != 128) return RMM_ERR_UNSUPPORTED;
    if (!aligned16(Q) || !aligned16(Kc) || !aligned16(V) || !aligned16(Ot)) return RMM_ERR_UNSUPPORTED;
    if (Lq % 8 || ldot % 8 || reinterpret_cast<uintptr_t>(energy) % 8) return RMM_ERR_UNSUPPORTED;
    if (batch * H > kGridYZMax || (Lq + 255) / 256 * batch * H > kInt32Max) return RMM_ERR_UNSUPPORTED;
    const size_t need = rmm_attention_kmajor_workspace_size(batch, H, Lq, Lk, D, k);
    if (!workspace || workspace_bytes < need) return RMM_ERR_WORKSPACE_TOO_SMALL;
    if (reinterpret_cast<uintptr_t>(workspace) % 256) return RMM_ERR_INVALID_ARGUMENT;
    char *ws = static_cast<char *>(workspace);
    uint16_t *Ki = reinterpret_cast<uint16_t *>(ws);
    double *partials = reinterpret_cast<double *>(ws + align256(rmm::attn_workspace_bytes(batch * H, Lk, k)));
    return from_hip(rmm::launch_attn_kmajor_bf16(
        static_cast<const uint16_t *>(Q), static_cast<const uint16_t *>(Kc),
        static_cast<const uint16_t *>(V), idx, batch, H, Hkv, Lq, Lk, k, scale, causal != 0,
        static_cast<uint16_t *>(Ot), ldot, energy, Ki, partials, stream));
}

rmm_status_t rmm_linear(const void *X, const void *W, double r, rmm_dtype_t dtype, int64_t B,
                        int64_t M, int64_t N, int64_t K, int64_t ldx, int64_t ldw, void *Y,
                        int64_t ldy, int32_t *idx_out, void *workspace, size_t workspace_bytes,
                        hipStream_t stream) {
    const int64_t k = rmm_retained_count(r, K);
    if (k < 0) return RMM_ERR_INVALID_ARGUMENT;
    rmm_status_t st = check_gemm_shapes(X, W, dtype, B, M, N, K, k, ldx, ldw, Y, ldy);
    if (st != RMM_OK) return st;
    const size_t need = rmm_workspace_size(RMM_OP_LINEAR, B, M, K, k);
    if (!workspace || workspace_bytes < need) return RMM_ERR_WORKSPACE_TOO_SMALL;
    if (reinterpret_cast<uintptr_t>(workspace) % 8) return RMM_ERR_INVALID_ARGUMENT;

    char *ws = static_cast<char *>(workspace);
    double *partials = reinterpret_cast<double *>(ws);
    ws += align256(rmm::score_workspace_bytes(B, M, K));
    double *energy = reinterpret_cast<double *>(ws);
    ws += align256(static_cast<size_t>(B * K) * sizeof(double));
    int32_t *idx = idx_out ? idx_out : reinterpret_cast<int32_t *>(ws);
    ws += align256(static_cast<size_t>(B * k) * sizeof(int32_t));
    uint16_t *Xt = reinterpret_cast<uint16_t *>(ws);

    // bf16 with 16-byte aligned rows: the scoring pass also writes the K-major
    // copy that the K-major GEMM gathers rows from
    const bool kmajor = dtype == RMM_BF16 && aligned16(X) && ldx % 8 == 0 && aligned16(Xt) &&
                        kmajor_ok(Xt, W, B, M, K, xt_ld(M), ldw);
    hipError_t e = rmm::launch_score(X, dtype == RMM_BF16, B, M, K, ldx, energy, partials,
                                     kmajor ? Xt : nullptr, xt_ld(M), stream);
    if (e != hipSuccess) return RMM_ERR_HIP;
    e = rmm::launch_select(energy, B, K, k, idx, stream);
    if (e != hipSuccess) return RMM_ERR_HIP;
    if (kmajor)
        e = rmm::launch_gemm_kmajor_bf16(Xt, static_cast<const uint16_t *>(W), idx, B, M, N, K, k,
                                         xt_ld(M), ldw, static_cast<uint16_t *>(Y), ldy, stream);
    else if (dtype == RMM_BF16)
        e = rmm::launch_gemm_bf16(static_cast<const uint16_t *>(X), static_cast<const uint16_t *>(W),
                                  idx, B, M, N, K, k, ldx, ldw, static_cast<uint16_t *>(Y), ldy,
                                  stream);
    else
        e = rmm::launch_gemm_f32(static_cast<const float *>(X), static_cast<const float *>(W), idx,
                                 B, M, N, K, k, ldx, ldw, static_cast<float *>(Y), ldy, stream);
    return from_hip(e);
}

rmm_status_t rmm_reduced_pv(const void *P, const void *V, rmm_dtype_t dtype, int64_t batch,
                            int64_t H, int64_t Hkv, int64_t Lq, int64_t Lk, int64_t D, int64_t ldp,
                            int64_t kt, void *O, int32_t *idx_out, void *workspace,
                            size_t workspace_bytes, hipStream_t stream) {
    if (!P || !V || !O) return RMM_ERR_INVALID_ARGUMENT;
    if (batch < 1 || H < 1 || Hkv < 1 || Lq < 1 || Lk < 1 || D < 1) return RMM_ERR_INVALID_ARGUMENT;
    if (H % Hkv != 0) return RMM_ERR_INVALID_ARGUMENT;
    const int64_t U = batch * H, grp = H / Hkv;
    // one product per (sequence, kv head): its query heads' units against V
    rmm_status_t st = check_gemm_shapes(P, V, dtype, grp, Lq, D, Lk, kt, ldp, D, O, D);
    if (st != RMM_OK) return st;
    if (U > kGridYZMax) return RMM_ERR_UNSUPPORTED;
    const size_t need = rmm_workspace_size(RMM_OP_PV, U, Lq, Lk, kt);
    if (!workspace || workspace_bytes < need) return RMM_ERR_WORKSPACE_TOO_SMALL;
    if (reinterpret_cast<uintptr_t>(workspace) % 8) return RMM_ERR_INVALID_ARGUMENT;

    char *ws = static_cast<char *>(workspace);
    double *partials = reinterpret_cast<double *>(ws);
    ws += align256(rmm::score_workspace_bytes(U, Lq, Lk));
    double *energy = reinterpret_cast<double *>(ws);
    ws += align256(static_cast<size_t>(U * Lk) * sizeof(double));
    int32_t *idx = idx_out ? idx_out : reinterpret_cast<int32_t *>(ws);
    ws += align256(static_cast<size_t>(U * kt) * sizeof(int32_t));
    uint16_t *Pt = reinterpret_cast<uint16_t *>(ws);

    // token energies of every head (column sums of P^2 over its queries),
    // with the K-major copy of P for bf16, then every head's TopK
    const bool bf16 = dtype == RMM_BF16;
    const bool kmajor = bf16 && aligned16(P) && ldp % 8 == 0 && aligned16(Pt) &&
                        kmajor_ok(Pt, V, grp, Lq, Lk, xt_ld(Lq), D);
    hipError_t e = rmm::launch_score(P, bf16, U, Lq, Lk, ldp, energy, partials,
                                     kmajor ? Pt : nullptr, xt_ld(Lq), stream);
    if (e != hipSuccess) return RMM_ERR_HIP;
    e = rmm::launch_select(energy, U, Lk, kt, idx, stream);
    if (e != hipSuccess) return RMM_ERR_HIP;
    const size_t esz = bf16 ? 2 : 4;
    if (kmajor) {
        // one launch over every query head, each reading its kv head's rows of V
        e = rmm::launch_gemm_kmajor_grouped_bf16(Pt, static_cast<const uint16_t *>(V), idx, U, Lq, D,
                                                 Lk, kt, xt_ld(Lq), D, static_cast<uint16_t *>(O), D,
                                                 Lk * D, static_cast<int>(grp), 0, 0, stream);
        return e == hipErrorNotSupported ? RMM_ERR_UNSUPPORTED : from_hip(e);
    }
    for (int64_t b = 0; b < batch && e == hipSuccess; ++b)
        for (int64_t g = 0; g < Hkv && e == hipSuccess; ++g) {
            const int64_t u0 = b * H + g * grp;
            const char *Vg = static_cast<const char *>(V) + (b * Hkv + g) * Lk * D * esz;
            char *Og = static_cast<char *>(O) + u0 * Lq * D * esz;
            const int32_t *ig = idx + u0 * kt;
            if (kmajor)
                e = rmm::launch_gemm_kmajor_bf16(Pt + u0 * Lk * xt_ld(Lq), reinterpret_cast<const uint16_t *>(Vg),
                                                 ig, grp, Lq, D, Lk, kt, xt_ld(Lq), D,
                                                 reinterpret_cast<uint16_t *>(Og), D, stream);
            else if (bf16)
                e = rmm::launch_gemm_bf16(static_cast<const uint16_t *>(P) + u0 * Lq * ldp,
                                          reinterpret_cast<const uint16_t *>(Vg), ig, grp, Lq, D, Lk, kt,
                                          ldp, D, reinterpret_cast<uint16_t *>(Og), D, stream);
            else
                e = rmm::launch_gemm_f32(static_cast<const float *>(P) + u0 * Lq * ldp,
                                         reinterpret_cast<const float *>(Vg), ig, grp, Lq, D, Lk, kt,
                                         ldp, D, reinterpret_cast<float *>(Og), D, stream);
        }
    return from_hip(e);
}

size_t rmm_attention_weights_kmajor_workspace_size(int64_t batch, int64_t H, int64_t Lq, int64_t Lk) {
    if (batch < 1 || H < 1 || Lq < 1 || Lk < 1) return 0;
    return align256(rmm::weights_workspace_bytes(batch * H, Lq, Lk));
}

static rmm_status_t attention_weights(const void *S, int64_t batch, int64_t H, int64_t Lq, int64_t Lk,
                                      int64_t lds, int causal, const float *row_max,
                                      const float *row_rinv, void *Pt, int64_t ldpt, double *energy,
                                      void *workspace, size_t workspace_bytes, hipStream_t stream) {
    if (!S || !Pt || !energy) return RMM_ERR_INVALID_ARGUMENT;
    if (batch < 1 || H < 1 || Lq < 1 || Lk < 1 || lds < Lk || ldpt < Lq) return RMM_ERR_INVALID_ARGUMENT;
    if (Lq > kInt32Max || Lk > kInt32Max) return RMM_ERR_INVALID_ARGUMENT;
    const int64_t U = batch * H;
    if (U > kGridYZMax) return RMM_ERR_UNSUPPORTED;
    if (!aligned16(S) || !aligned16(Pt) || lds % 8 || ldpt % 8 ||
        reinterpret_cast<uintptr_t>(energy) % 8)
        return RMM_ERR_UNSUPPORTED;
    // the tile kernel addresses one row split with 32-bit byte offsets
    if (rmm::score_rows_per_split(U, Lq, Lk) * lds * 2 >= (int64_t(1) << 31)) return RMM_ERR_UNSUPPORTED;
    const size_t need = rmm_attention_weights_kmajor_workspace_size(batch, H, Lq, Lk);
    if (!workspace || workspace_bytes < need) return RMM_ERR_WORKSPACE_TOO_SMALL;
    if (reinterpret_cast<uintptr_t>(workspace) % 256) return RMM_ERR_INVALID_ARGUMENT;
    return from_hip(rmm::launch_attention_weights_kmajor(
        static_cast<const uint16_t *>(S), U, Lq, Lk, lds, causal != 0, row_max, row_rinv,
        static_cast<uint16_t *>(Pt), ldpt, energy, workspace, stream));
}

rmm_status_t rmm_attention_weights_kmajor(const void *S, int64_t batch, int64_t H, int64_t Lq,
                                          int64_t Lk, int64_t lds, int causal, void *Pt,
                                          int64_t ldpt, double *energy, void *workspace,
                                          size_t workspace_bytes, hipStream_t stream) {
    return attention_weights(S, batch, H, Lq, Lk, lds, causal, nullptr, nullptr, Pt, ldpt, energy,
                             workspace, workspace_bytes, stream);
}

rmm_status_t rmm_attention_weights_kmajor_rowstats(const void *S, int64_t batch, int64_t H, int64_t Lq,
                                                   int64_t Lk, int64_t lds, int causal,
                                                   const float *row_max, const float *row_rinv,
                                                   void *Pt, int64_t ldpt, double *energy,
                                                   void *workspace, size_t workspace_bytes,
                                                   hipStream_t stream) {
    if (!row_max || !row_rinv) return RMM_ERR_INVALID_ARGUMENT;
    if (reinterpret_cast<uintptr_t>(row_max) % 4 || reinterpret_cast<uintptr_t>(row_rinv) % 4)
        return RMM_ERR_UNSUPPORTED;
    return attention_weights(S, batch, H, Lq, Lk, lds, causal, row_max, row_rinv, Pt, ldpt, energy,
                             workspace, workspace_bytes, stream);
}

rmm_status_t rmm_reduced_pv_kmajor(const void *Pt, const void *V, const int32_t *idx, int64_t batch,
                                   int64_t H, int64_t Hkv, int64_t Lq, int64_t Lk, int64_t D,
                                   int64_t kt, int64_t ldpt, int causal, void *O, hipStream_t stream) {
    if (!Pt || !V || !idx || !O) return RMM_ERR_INVALID_ARGUMENT;
    if (batch < 1 || H < 1 || Hkv < 1 || Lq < 1 || Lk < 1 || D < 1) return RMM_ERR_INVALID_ARGUMENT;
    if (H % Hkv != 0 || kt < 1 || kt > Lk || ldpt < Lq) return RMM_ERR_INVALID_ARGUMENT;
    if (Lq > kInt32Max || Lk > kInt32Max || D > kInt32Max) return RMM_ERR_INVALID_ARGUMENT;
    const int64_t U = batch * H, grp = H / Hkv;
    if (U > kGridYZMax || !kmajor_ok(Pt, V, U, Lq, Lk, ldpt, D)) return RMM_ERR_UNSUPPORTED;
    const uint16_t *pt = static_cast<const uint16_t *>(Pt), *v = static_cast<const uint16_t *>(V);
    uint16_t *o = static_cast<uint16_t *>(O);
    // one launch over every query head; with the causal mask each row tile
    // stops at the last kept token any of its queries can see
    const hipError_t e = rmm::launch_gemm_kmajor_grouped_bf16(
        pt, v, idx, U, Lq, D, Lk, kt, ldpt, D, o, D, Lk * D, static_cast<int>(grp), causal != 0, Lk - Lq,
        stream);
    return e == hipErrorNotSupported ? RMM_ERR_UNSUPPORTED : from_hip(e);
}

// The grouped decode step's kernel arguments from the caller's groups (shapes
// validated), with each group's partials carved from the workspace when ws is
// given; returns the workspace bytes needed.
static size_t decode_groups(const rmm_decode_group_t *groups, int n, int64_t B, void *ws,
                            rmm::GemvGroups *G) {
    size_t off = 0;
    G->n = n;
    for (int i = 0; i < n; ++i) {
        const rmm_decode_group_t &d = groups[i];
        rmm::GemvGroup &q = G->g[i];
        q.X = static_cast<const uint16_t *>(d.X);
        q.W = static_cast<const uint16_t *>(d.W);
        q.idx = d.idx;
        q.idx_out = d.idx;
        q.Y = static_cast<uint16_t *>(d.Y);
        q.N = static_cast<int>(d.N);
        q.K = static_cast<int>(d.K);
        q.k = static_cast<int>(d.k);
        q.ldx = d.ldx;
        q.ldw = d.ldw;
        q.ldy = d.ldy;
        int SR, S;
        rmm::gemv_slices(B, d.N, d.k, &SR, &S);
        q.P = (S > 1 && ws) ? reinterpret_cast<float *>(static_cast<char *>(ws) + off) : nullptr;
        if (S > 1) off += align256(static_cast<size_t>(B) * S * d.N * sizeof(float));
    }
    return off;
}

static rmm_status_t check_decode_groups(const rmm_decode_group_t *groups, int n, int64_t B) {
    if (!groups || n < 1 || B < 1) return RMM_ERR_INVALID_ARGUMENT;
    if (n > rmm::kMaxGemvGroups || B > kGridYZMax) return RMM_ERR_UNSUPPORTED;
    for (int i = 0; i < n; ++i) {
        const rmm_decode_group_t &d = groups[i];
        if (!d.X || !d.W || !d.idx || !d.Y) return RMM_ERR_INVALID_ARGUMENT;
        if (d.K < 1 || d.N < 1 || d.k < 1 || d.k > d.K) return RMM_ERR_INVALID_ARGUMENT;
        if (d.ldx < d.K || d.ldw < d.N || d.ldy < d.N) return RMM_ERR_INVALID_ARGUMENT;
        if (d.N > kInt32Max) return RMM_ERR_INVALID_ARGUMENT;
        if (!aligned16(d.X) || d.ldx % 8 || !aligned16(d.W) || d.ldw % 8)
            return RMM_ERR_UNSUPPORTED;
        if (d.K * d.ldw * 2 >= (int64_t(1) << 31)) return RMM_ERR_UNSUPPORTED;
    }
    return RMM_OK;
}

size_t rmm_decode_step_workspace_size(const rmm_decode_group_t *groups, int ngroups, int64_t B) {
    if (check_decode_groups(groups, ngroups, B) != RMM_OK) return 0;
    rmm::GemvGroups G;
    return decode_groups(groups, ngroups, B, nullptr, &G);
}

rmm_status_t rmm_decode_step(const rmm_decode_group_t *groups, int ngroups, int64_t B,
                             void *workspace, size_t workspace_bytes, hipStream_t stream) {
    rmm_status_t st = check_decode_groups(groups, ngroups, B);
    if (st != RMM_OK) return st;
    rmm::GemvGroups G;
    const size_t need = decode_groups(groups, ngroups, B, nullptr, &G);
    if (need > 0) {
        if (!workspace || workspace_bytes < need) return RMM_ERR_WORKSPACE_TOO_SMALL;
        if (reinterpret_cast<uintptr_t>(workspace) % 256) return RMM_ERR_INVALID_ARGUMENT;
    }
    decode_groups(groups, ngroups, B, workspace, &G);
    hipError_t e = rmm::launch_select_tokens_grouped(G, B, stream);
    if (e != hipSuccess) return RMM_ERR_HIP;
    return from_hip(rmm::launch_gemv_grouped_bf16(G, B, stream));
}

rmm_status_t rmm_decode_products(const rmm_decode_group_t *groups, int ngroups, int64_t B,
                                 void *workspace, size_t workspace_bytes, hipStream_t stream) {
    rmm_status_t st = check_decode_groups(groups, ngroups, B);
    if (st != RMM_OK) return st;
    rmm::GemvGroups G;
    const size_t need = decode_groups(groups, ngroups, B, nullptr, &G);
    if (need > 0) {
        if (!workspace || workspace_bytes < need) return RMM_ERR_WORKSPACE_TOO_SMALL;
        if (reinterpret_cast<uintptr_t>(workspace) % 256) return RMM_ERR_INVALID_ARGUMENT;
    }
    decode_groups(groups, ngroups, B, workspace, &G);
    return from_hip(rmm::launch_gemv_grouped_bf16(G, B, stream));
}

// The shared-rows decode products' kernel arguments (shapes validated), each
// group's workspace carved from ws; returns the workspace bytes needed.
static size_t share_groups(const rmm_decode_group_t *groups, int n, int64_t B, void *ws,
                           rmm::ShareGroups *G) {
    size_t off = 0;
    G->n = n;
    for (int i = 0; i < n; ++i) {
        const rmm_decode_group_t &d = groups[i];
        rmm::ShareGroup &q = G->g[i];
        q = rmm::ShareGroup{};
        q.X = static_cast<const uint16_t *>(d.X);
        q.W = static_cast<const uint16_t *>(d.W);
        q.idx = d.idx;
        q.Y = static_cast<uint16_t *>(d.Y);
        q.N = static_cast<int>(d.N);
        q.K = static_cast<int>(d.K);
        q.k = static_cast<int>(d.k);
        q.ldx = d.ldx;
        q.ldw = d.ldw;
        q.ldy = d.ldy;
        void *base = ws ? static_cast<void *>(static_cast<char *>(ws) + off) : nullptr;
        off += align256(rmm::share_group_layout(B, d.N, d.K, base, &q));
    }
    return off;
}

static rmm_status_t check_share_groups(const rmm_decode_group_t *groups, int n, int64_t B) {
    const rmm_status_t st = check_decode_groups(groups, n, B);
    if (st != RMM_OK) return st;
    return B > rmm::kShareMaxB ? RMM_ERR_UNSUPPORTED : RMM_OK;
}

size_t rmm_decode_products_shared_workspace_size(const rmm_decode_group_t *groups, int ngroups,
                                                 int64_t B) {
    if (check_share_groups(groups, ngroups, B) != RMM_OK) return 0;
    rmm::ShareGroups G;
    return share_groups(groups, ngroups, B, nullptr, &G);
}

rmm_status_t rmm_decode_products_shared(const rmm_decode_group_t *groups, int ngroups, int64_t B,
                                        void *workspace, size_t workspace_bytes, hipStream_t stream) {
    const rmm_status_t st = check_share_groups(groups, ngroups, B);
    if (st != RMM_OK) return st;
    rmm::ShareGroups G;
    const size_t need = share_groups(groups, ngroups, B, nullptr, &G);
    if (!workspace || workspace_bytes < need) return RMM_ERR_WORKSPACE_TOO_SMALL;
    if (reinterpret_cast<uintptr_t>(workspace) % 256) return RMM_ERR_INVALID_ARGUMENT;
    share_groups(groups, ngroups, B, workspace, &G);
    return from_hip(rmm::launch_share_products(G, B, stream));
}

rmm_status_t rmm_decode_step_shared(const rmm_decode_group_t *groups, int ngroups, int64_t B,
                                    void *workspace, size_t workspace_bytes, hipStream_t stream) {
    const rmm_status_t st = check_share_groups(groups, ngroups, B);
    if (st != RMM_OK) return st;
    rmm::ShareGroups G;
    const size_t need = share_groups(groups, ngroups, B, nullptr, &G);
    if (!workspace || workspace_bytes < need) return RMM_ERR_WORKSPACE_TOO_SMALL;
    if (reinterpret_cast<uintptr_t>(workspace) % 256) return RMM_ERR_INVALID_ARGUMENT;
    // the selection reads the tokens and writes the lists (no workspace)
    rmm::GemvGroups S;
    decode_groups(groups, ngroups, B, nullptr, &S);
    if (rmm::launch_select_tokens_grouped(S, B, stream) != hipSuccess) return RMM_ERR_HIP;
    share_groups(groups, ngroups, B, workspace, &G);
    return from_hip(rmm::launch_share_products(G, B, stream));
}

const char *rmm_status_string(rmm_status_t status) {
    switch (status) {
    case RMM_OK: return "success";
    case RMM_ERR_INVALID_ARGUMENT: return "invalid argument";
    case RMM_ERR_UNSUPPORTED: return "unsupported argument combination";
    case RMM_ERR_WORKSPACE_TOO_SMALL: return "workspace missing or too small";
    case RMM_ERR_HIP: return "HIP launch failed";
    case RMM_ERR_TOO_LARGE: return "problem exceeds the library's fixed scratch buffer";
    }
    return "unknown status";
}

}  // extern "C"
