// Internal launchers of librmm's gfx950 kernels.  Arguments are validated by
// the C-ABI layer (api.hip) before any of these is called.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rmm {

// ---------------------------------------------------------------- scoring
// Column energies are reduced in two levels: a grid of (column block, row
// split, unit) workgroups writes float64 partial sums, then a second kernel
// adds the splits in a fixed order.  Splits depend only on (B, M, K).
constexpr int kScoreCols = 128;        // columns per workgroup
constexpr int kScoreMinRows = 64;      // fewest rows per split
constexpr int kScoreTargetBlocks = 2048;

int64_t score_rows_per_split(int64_t B, int64_t M, int64_t K);
// energy[b][j] = sum over s = 0..S-1, in order, of partials[b][s][j]
hipError_t launch_score_finalize(const double *partials, int64_t B, int64_t S, int64_t K,
                                 double *energy, hipStream_t stream);
// the same sum for many splits (a fixed order of its own: 16 consecutive
// runs of splits, each in order, then the runs in order)
hipError_t launch_score_finalize_grouped(const double *partials, int64_t B, int64_t S, int64_t K,
                                         double *energy, hipStream_t stream);
int64_t score_splits(int64_t B, int64_t M, int64_t K);
size_t score_workspace_bytes(int64_t B, int64_t M, int64_t K);

// Xt (nullable): also write the K-major copy Xt[b][j][m] (bf16 only, X rows
// 16-byte aligned, Xt 16-byte aligned with ldxt % 8 == 0).
hipError_t launch_score(const void *X, bool bf16, int64_t B, int64_t M, int64_t K,
                        int64_t ldx, double *energy, double *partials, uint16_t *Xt,
                        int64_t ldxt, hipStream_t stream);

// The scoring pass over RMSNorm-normalised rows: y = bf16(gamma_j *
// bf16(x * rscale[m])) (rscale [B][M] floats), energies and K-major copy of y
// (bf16, 16-byte aligned rows, as for the K-major scoring pass)
hipError_t launch_score_norm_kmajor(const uint16_t *X, int64_t B, int64_t M, int64_t K, int64_t ldx,
                                   const float *rscale, const uint16_t *gamma, double *energy,
                                   double *partials, uint16_t *Xt, int64_t ldxt, hipStream_t stream);
// RMSNorm writing the K-major normalised activations and their column
// energies (bf16, K % 8 == 0, 16-byte aligned rows; checked by the caller);
// the workspace (rmsnorm_workspace_bytes, 256-byte aligned, enough for
// either path) holds the partial energies (and, for rows wider than one pass
// takes, the row scales); rmsnorm_single_pass: whether rows of K channels at
// stride ldx are normalised in one pass
bool rmsnorm_single_pass(int64_t K, int64_t ldx);
size_t rmsnorm_workspace_bytes(int64_t B, int64_t M, int64_t K);
hipError_t launch_rmsnorm_kmajor(const uint16_t *X, const uint16_t *gamma, float eps, int64_t B,
                                 int64_t M, int64_t K, int64_t ldx, uint16_t *Xt, int64_t ldxt,
                                 double *energy, void *workspace, hipStream_t stream);

// -------------------------------------------------------------- selection
// TopK of x_j^2 for units of one token (row b of X at b * ldx)
hipError_t launch_select_tokens(const void *X, bool bf16, int64_t B, int64_t K, int64_t ldx,
                                int64_t k, int32_t *idx, hipStream_t stream);
hipError_t launch_select(const double *energy, int64_t B, int64_t K, int64_t k,
                         int32_t *idx, hipStream_t stream);
// bad[b]: 0 if unit b's list is strictly ascending within [0, K), else 1 + the
// first position that breaks it
hipError_t launch_check_indices(const int32_t *idx, int64_t B, int64_t k, int64_t K, int32_t *bad,
                                hipStream_t stream);

// ------------------------------------------------------- gathered GEMM
hipError_t launch_gemm_bf16(const uint16_t *X, const uint16_t *W, const int32_t *idx,
                            int64_t B, int64_t M, int64_t N, int64_t K, int64_t k,
                            int64_t ldx, int64_t ldw, uint16_t *Y, int64_t ldy,
                            hipStream_t stream);
// Xt: K-major activations [B][K][ldxt]; 16-byte aligned, ldxt % 8 == 0,
// K*ldxt*2 and K*ldw*2 below 2^31 (checked by the caller).
hipError_t launch_gemm_kmajor_bf16(const uint16_t *Xt, const uint16_t *W, const int32_t *idx,
                                  int64_t B, int64_t M, int64_t N, int64_t K, int64_t k,
                                  int64_t ldxt, int64_t ldw, uint16_t *Y, int64_t ldy,
                                  hipStream_t stream);
// the same product with per-unit weights: unit u reads W + (u / w_ugroup) *
// w_ustride elements; with trim, Xt is known to be zero at (m, j) for
// j > m + trim_off and each row tile stops its K loop there;
// hipErrorNotSupported (nothing launched) when ldy >= 2^23 (the large-tile
// kernel that implements these addresses Y rows with 32-bit offsets)
hipError_t launch_gemm_kmajor_grouped_bf16(const uint16_t *Xt, const uint16_t *W, const int32_t *idx,
                                          int64_t B, int64_t M, int64_t N, int64_t K, int64_t k,
                                          int64_t ldxt, int64_t ldw, uint16_t *Y, int64_t ldy,
                                          int64_t w_ustride, int w_ugroup, int trim, int64_t trim_off,
                                          hipStream_t stream);
// the transposing scoring pass over attention scores: Pt = the K-major
// softmax weights exp(s - rmax[m]) * rinv[m] (zero where causal drops j > m +
// coff), and their column energies
hipError_t launch_score_softmax_kmajor(const uint16_t *S, int64_t B, int64_t M, int64_t K, int64_t ld,
                                      const float *rmax, const float *rinv, int64_t coff,
                                      int causal, double *energy, double *partials, uint16_t *Pt,
                                      int64_t ldpt, hipStream_t stream);
// softmax weights of attention scores written K-major with their token
// energies (bf16 S rows 16-byte aligned; checked by the caller); the
// workspace (weights_workspace_bytes, 256-byte aligned) holds the row
// statistics and the scoring partials; with rmax_in and rinv_in given the
// row statistics are taken from them and not computed
size_t weights_workspace_bytes(int64_t U, int64_t Lq, int64_t Lk);
hipError_t launch_attention_weights_kmajor(const uint16_t *S, int64_t U, int64_t Lq, int64_t Lk,
                                           int64_t lds, int causal, const float *rmax_in,
                                           const float *rinv_in, uint16_t *Pt, int64_t ldpt,
                                           double *energy, void *workspace, hipStream_t stream);
// the gate|up product with the SwiGLU epilogue: W [K][ldw] holds 2F columns
// in 128-column blocks (gate, then up, of the same 128 channels); writes the
// down projection's K-major input Ht [B][F][ldht] and its column energies
// energy [B][F]; partials holds B * ceil(M/256) * F doubles.  F % 128 == 0,
// M % 8 == 0, ldht % 8 == 0, Ht 16-byte aligned (checked by the caller).
hipError_t launch_gemm_swiglu_kmajor_bf16(const uint16_t *Xt, const uint16_t *W,
                                         const int32_t *idx, int64_t B, int64_t M, int64_t F,
                                         int64_t K, int64_t k, int64_t ldxt, int64_t ldw,
                                         uint16_t *Ht, int64_t ldht, double *energy,
                                         double *partials, hipStream_t stream);
hipError_t launch_gemm_f32(const float *X, const float *W, const int32_t *idx,
                           int64_t B, int64_t M, int64_t N, int64_t K, int64_t k,
                           int64_t ldx, int64_t ldw, float *Y, int64_t ldy,
                           hipStream_t stream);

// Independent one-row-per-unit products of a decode step, passed by value
// to the grouped kernels (at most kMaxGemvGroups).  The launchers fill in
// the split (SR, S, chunks) and the workgroup numbering (first, rfirst).
constexpr int kMaxGemvGroups = 8;
struct GemvGroup {
    const uint16_t *X;      // [B][ldx] bf16, one token per unit
    const uint16_t *W;      // [K][ldw] bf16, 16-byte aligned, ldw % 8 == 0
    const int32_t *idx;     // [B][k] the retained lists the product reads
    int32_t *idx_out;       // [B][k] the lists the selection writes (same memory)
    uint16_t *Y;            // [B][ldy] bf16
    float *P;               // [B][S][N] fp32 partials when S > 1
    int N, K, k;
    int64_t ldx, ldw, ldy;
    int SR, S, chunks, first, rfirst;
};
struct GemvGroups {
    GemvGroup g[kMaxGemvGroups];
    int n;
};
// TopK of x^2 for every unit of every group (bf16 tokens, 16-byte aligned
// rows; checked by the caller): one launch for the groups of up to
// kToken16MaxK channels, one launch of the generic selection per wider group
constexpr int64_t kToken16MaxK = 32 * 1024;
hipError_t launch_select_tokens_grouped(const GemvGroups &G, int64_t B, hipStream_t stream);
// the groups' reduced products (one launch) and slice reductions (one launch)
hipError_t launch_gemv_grouped_bf16(GemvGroups G, int64_t B, hipStream_t stream);

// reduced product with M <= 8 rows per unit (decode); workspace holds the
// per-slice fp32 partials when the retained list is split
void gemv_slices(int64_t B, int64_t N, int64_t k, int *SR, int *S);
size_t gemv_workspace_bytes(int64_t B, int64_t M, int64_t N, int64_t k);
hipError_t launch_gemv_bf16(const uint16_t *X, const uint16_t *W, const int32_t *idx, int64_t B,
                            int64_t M, int64_t N, int64_t K, int64_t k, int64_t ldx, int64_t ldw,
                            uint16_t *Y, int64_t ldy, void *workspace, hipStream_t stream);

// --------------------------------------------------------- reduced QK^T
// reduced attention block, bf16, D == 128, 16-byte aligned (checked by the
// caller); the workspace holds the per-head compacted key rows
int attn_k_steps(int64_t k);
size_t attn_workspace_bytes(int64_t batch_heads, int64_t Lk, int64_t k);
hipError_t launch_attn_bf16(const uint16_t *Q, const uint16_t *Kc, const uint16_t *V,
                            const int32_t *idx, int64_t batch, int64_t H, int64_t Hkv,
                            int64_t Lq, int64_t Lk, int64_t k, float scale, bool causal,
                            uint16_t *O, void *workspace, hipStream_t stream);
// the same block writing its output as the K-major input of the following
// projection, Ot[b][h*D + j][ldot] (Lq % 8 == 0, ldot % 8 == 0, Ot 16-byte
// aligned), and that input's column energies energy[b][h*D + j]; partials
// holds batch * attn_query_tiles(Lq) * H * D doubles
int64_t attn_query_tiles(int64_t Lq);
hipError_t launch_attn_kmajor_bf16(const uint16_t *Q, const uint16_t *Kc, const uint16_t *V,
                                   const int32_t *idx, int64_t batch, int64_t H, int64_t Hkv,
                                   int64_t Lq, int64_t Lk, int64_t k, float scale, bool causal,
                                   uint16_t *Ot, int64_t ldot, double *energy, uint16_t *Ki,
                                   double *partials, hipStream_t stream);
hipError_t launch_qk_bf16(const uint16_t *Q, const uint16_t *Kc, const int32_t *idx,
                          int64_t batch, int64_t H, int64_t Hkv, int64_t Lq,
                          int64_t Lk, int64_t D, int64_t k, float scale, bool causal,
                          uint16_t *S, hipStream_t stream);
// the row-major bf16 scores with each row's softmax statistics over its
// stored kept scores (max, 1 / sum of exp(s - max); 0, 0 for an empty row);
// hipErrorNotSupported (nothing launched) unless qk_rows_ok
bool qk_rows_ok(int64_t Lk, int64_t D, const void *S);
hipError_t launch_qk_rowstats_bf16(const uint16_t *Q, const uint16_t *Kc, const int32_t *idx,
                                   int64_t batch, int64_t H, int64_t Hkv, int64_t Lq, int64_t Lk,
                                   int64_t D, int64_t k, float scale, bool causal, uint16_t *S,
                                   float *rmax, float *rinv, hipStream_t stream);
hipError_t launch_qk_f32(const float *Q, const float *Kc, const int32_t *idx,
                         int64_t batch, int64_t H, int64_t Hkv, int64_t Lq,
                         int64_t Lk, int64_t D, int64_t k, float scale, bool causal,
                         float *S, hipStream_t stream);

}  // namespace rmm
