/*
 * librmm -- Reduced Matrix Multiplication (RMM) on AMD Instinct MI355X (gfx950).
 *
 * RMM (arXiv 2608.13426, Sec. 3.2) replaces a product Y = A B, A in R^{n x d},
 * B in R^{d x m}, by A[:, I] B[I, :] where I holds the ceil(rho*d) indices of
 * the shared axis with the largest activation column norms ||A[:, j]||_2.
 * Sec. 3.3 applies it to linear / MLP projections (A = X, B = W) and, per
 * attention head, to Q K^T over the head dimension.
 *
 * Conventions shared by every entry point:
 *
 *  - All tensor pointers are DEVICE pointers unless stated otherwise.  The
 *    caller allocates and frees every buffer; the library never allocates
 *    device memory.  Scratch memory, where needed, is a caller-provided
 *    workspace sized by rmm_workspace_size().
 *  - Every call validates its arguments on the host first and returns
 *    RMM_ERR_INVALID_ARGUMENT / RMM_ERR_UNSUPPORTED / RMM_ERR_WORKSPACE_TOO_SMALL
 *    without touching the device.  Valid calls enqueue kernels on `stream`
 *    (NULL = the legacy default stream) and return without synchronising;
 *    RMM_ERR_HIP reports a failed launch.  Nothing is printed, nothing aborts.
 *  - Matrices are row-major with a leading dimension (elements between
 *    consecutive rows).  bf16 tensors hold raw bfloat16 bit patterns.
 *  - Arithmetic: energies are float64 sums of exact squares; bf16 products
 *    accumulate in fp32 and are rounded to bf16 (round-to-nearest-even) on
 *    output; the fp32 path accumulates and outputs fp32.
 *  - Index sets are int32, strictly ascending, one set per selection unit.
 *    Selection is deterministic: energy descending, ties to the lower index,
 *    NaN above +inf above every finite value.  No call uses floating-point
 *    atomics, so repeated calls give bit-identical results.
 *  - Calls are reentrant and may run concurrently on different streams with
 *    distinct output and workspace buffers.
 */
#ifndef RMM_H
#define RMM_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum rmm_status {
    RMM_OK = 0,
    RMM_ERR_INVALID_ARGUMENT = 1,   /* null pointer, bad size, r outside (0,1], ... */
    RMM_ERR_UNSUPPORTED = 2,        /* valid but not implemented (dtype, alignment) */
    RMM_ERR_WORKSPACE_TOO_SMALL = 3,
    RMM_ERR_HIP = 4,                /* a HIP launch failed (no device, bad stream) */
    RMM_ERR_TOO_LARGE = 5           /* exceeds the fixed scratch of rmm_linear_noalloc */
} rmm_status_t;

typedef enum rmm_dtype {
    RMM_F32 = 0,    /* float32 in, float32 out */
    RMM_BF16 = 1    /* bfloat16 in, fp32 accumulate, bfloat16 out */
} rmm_dtype_t;

typedef enum rmm_op {
    RMM_OP_SCORE = 0,   /* rmm_score   */
    RMM_OP_SELECT = 1,  /* rmm_select  */
    RMM_OP_LINEAR = 2,  /* rmm_linear  */
    RMM_OP_ATTENTION = 3, /* rmm_reduced_attention */
    RMM_OP_PV = 4         /* rmm_reduced_pv */
} rmm_op_t;

/*
 * Number of retained indices k = ceil(r * K)   (Sec. 3.2: |I| = ceil(rho d)).
 *
 * r is read as the decimal the caller meant: when r*K lies within 1e-9*K of
 * an integer that integer is k (so r = 0.07, K = 100 gives 7, not 8).  The
 * result is clamped to [1, K].  Host-only; returns -1 when r is not in
 * (0, 1] (or is NaN), when K < 1, or when K > INT32_MAX.
 */
int64_t rmm_retained_count(double r, int64_t K);

/*
 * Bytes of workspace a call needs (0 if none).  Arguments as in the call:
 *   RMM_OP_SCORE : B, M, K        (k ignored)
 *   RMM_OP_SELECT: always 0
 *   RMM_OP_LINEAR: B, M, K, k     (k = rmm_retained_count(r, K); includes
 *                  room for the K-major copy of X, B*K*round_up(M, 8) bf16)
 *   RMM_OP_ATTENTION: B = batch*H, M = Lk, K = D, k  (each query head's
 *                  retained key dims as rows: B*Lk*kp bf16, kp = k rounded
 *                  up to 32, 64, 96 or 128)
 *   RMM_OP_PV    : B = batch*H, M = Lq, K = Lk, k = kt (as RMM_OP_LINEAR)
 * Returns 0 for non-positive sizes.  Host-only.
 */
size_t rmm_workspace_size(rmm_op_t op, int64_t B, int64_t M, int64_t K, int64_t k);

/*
 * Column energies   (Sec. 3.2, score s_j = ||A[:, j]||_2; Sec. 3.3 for Q).
 *
 *   energy[b*K + j] = sum_{m < M} X[b][m][j]^2          (= s_j^2)
 *
 * X        : B selection units, each M rows of K values, row stride ldx
 *            (ldx >= K), unit stride M*ldx.  For attention scores pass Q
 *            [batch*H][Lq][D] with B = batch*H, M = Lq, K = ldx = D.
 * dtype    : RMM_BF16 or RMM_F32.
 * energy   : float64 [B*K], written.  Squares are exact; the sum is float64
 *            in a fixed order that depends only on (B, M, K).  NaN/Inf
 *            inputs propagate into the energies.
 * workspace: rmm_workspace_size(RMM_OP_SCORE, B, M, K, 0) bytes, 8-byte
 *            aligned (may be NULL when that size is 0).
 * Errors   : INVALID_ARGUMENT for null pointers, B/M/K < 1, ldx < K, K >
 *            INT32_MAX, a misaligned workspace; UNSUPPORTED for B > 65535;
 *            WORKSPACE_TOO_SMALL.
 */
rmm_status_t rmm_score(const void *X, rmm_dtype_t dtype, int64_t B, int64_t M,
                       int64_t K, int64_t ldx, double *energy,
                       void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Column energies plus a K-major copy of the activations   (Sec. 3.2 score;
 * the copy feeds rmm_reduced_gemm_kmajor).
 *
 * Computes exactly what rmm_score computes for bf16 (bit-identical energies)
 * and, in the same pass over X, writes Xt[b][j][m] = X[b][m][j]: unit b's
 * K x M transpose, row stride ldxt (ldxt >= M).  A retained index j is then
 * one contiguous row of Xt.  bf16 only.
 *
 * X        : [B][M][ldx] bf16, 16-byte aligned, ldx % 8 == 0.
 * Xt       : [B][K][ldxt] bf16, written; 16-byte aligned, ldxt % 8 == 0.
 * energy, workspace: as rmm_score (same workspace size).
 * Errors   : as rmm_score; INVALID_ARGUMENT for a null Xt or ldxt < M;
 *            UNSUPPORTED for misaligned X/Xt or ldx, ldxt not multiples of 8.
 */
rmm_status_t rmm_score_kmajor(const void *X, int64_t B, int64_t M, int64_t K, int64_t ldx,
                              double *energy, void *Xt, int64_t ldxt,
                              void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * RMSNorm producing a reduced projection's input, K-major, with its column
 * energies   (Sec. 3.2: the retained set is scored on the projection's own
 * input; Sec. 3.3 reduces the attention and MLP projections, whose inputs
 * the LLaMA-family models produce with RMSNorm; the Limitations section
 * names the memory movement of a separate scoring pass as a cost to remove).
 *
 * For each unit b and row m of X (bf16):
 *   r_m          = 1 / sqrt(mean_j X[b][m][j]^2 + eps)      (fp32)
 *   y[m][j]      = bf16(gamma[j] * bf16(X[b][m][j] * r_m))   (the model's
 *                  normalised value, rounded as its bf16 output, times the
 *                  weight, rounded again)
 *   Xt[b][j][m]  = y[m][j]                                    (K-major)
 *   energy[b][j] = sum over m < M of y[m][j]^2                (float64 sums
 *                  of exact squares in a fixed order)
 * which is what rmm_score_kmajor would compute on the normalised rows,
 * without writing them row-major first: feed them to rmm_select and
 * rmm_reduced_gemm_kmajor.
 *
 * X     : bf16 [B][M][ldx], ldx >= K.      gamma : bf16 [K] (the norm weight).
 * Xt    : bf16 [B][K][ldxt], ldxt >= M; columns M..ldxt-1 are not written.
 * energy: float64 [B][K].   eps >= 0 (finite).
 * workspace : rmm_rmsnorm_kmajor_workspace_size(B, M, K) bytes, 256-byte
 *         aligned (row scales and partial energies; overwritten by every call).
 * Errors: INVALID_ARGUMENT for null pointers, sizes < 1, ldx < K, ldxt < M,
 *         eps negative, infinite or NaN, a misaligned workspace; UNSUPPORTED
 *         unless K % 8 == 0, B <= 65535, X, gamma and Xt are 16-byte aligned
 *         and ldx, ldxt are multiples of 8; WORKSPACE_TOO_SMALL.
 */
size_t rmm_rmsnorm_kmajor_workspace_size(int64_t B, int64_t M, int64_t K);
rmm_status_t rmm_rmsnorm_kmajor(const void *X, const void *gamma, float eps, int64_t B, int64_t M,
                                int64_t K, int64_t ldx, void *Xt, int64_t ldxt, double *energy,
                                void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * TopK selection   (Sec. 3.2: I = TopK({s_j}, ceil(rho d))).
 *
 * For each unit b, writes the k indices of the largest energy[b*K + j] to
 * idx[b*k .. b*k + k) in ascending order.  Order: larger energy first; equal
 * energies (including -0 == +0) go to the lower index; any NaN ranks above
 * +inf and NaNs tie with each other.  Integer-exact: the result depends
 * only on the float64 values passed in.
 *
 * energy : float64 [B*K] (device).        idx : int32 [B*k] (device), written.
 * Errors : INVALID_ARGUMENT for null pointers, B < 1, K < 1, k outside [1, K],
 *          K > INT32_MAX.
 */
rmm_status_t rmm_select(const double *energy, int64_t B, int64_t K, int64_t k,
                        int32_t *idx, hipStream_t stream);

/*
 * Selection for units of one token   (Sec. 3.2 TopK of the column norms;
 * App. A: in a decode step the set follows the current token).
 *
 * For B units of a single row each (one token per sequence), idx[b] is the
 * list rmm_score + rmm_select give for M = 1: the k indices with the largest
 * x_j^2 = X[b][j]^2, ties to the lower index, NaN above +inf above every
 * finite value, -0 == +0, ascending.  x_j^2 is exact in float64 and orders
 * like |x_j|, so the keys are taken from the activations directly: one
 * launch, no energies written.
 *
 * X   : [B][ldx] bf16 or fp32 (ldx >= K).    idx : int32 [B*k].
 * Errors: INVALID_ARGUMENT for null pointers, an unknown dtype, B < 1,
 *         K < 1, k outside [1, K], ldx < K, K > INT32_MAX.
 */
rmm_status_t rmm_select_tokens(const void *X, rmm_dtype_t dtype, int64_t B, int64_t K,
                               int64_t ldx, int64_t k, int32_t *idx, hipStream_t stream);

/*
 * Index-list check   (Sec. 3.2: I is a subset of [d] of size k; the gathered
 * products take any such list, e.g. the static variant or the random
 * selection that Sec. 4 "Baselines" compares against, as caller-made lists).
 *
 * bad[b] = 0 when idx[b*k .. b*k + k) is strictly ascending with every value
 * in [0, K) -- the precondition of rmm_reduced_gemm, rmm_reduced_gemm_kmajor,
 * rmm_reduced_gemv, rmm_reduced_qk and the attention entry points -- else
 * 1 + the first position t that breaks it (idx[t] outside [0, K) or
 * idx[t] <= idx[t-1]).  Lists made by rmm_select / rmm_select_tokens always
 * pass.
 * idx : int32 [B*k] (device).   bad : int32 [B] (device), written.
 * Errors: INVALID_ARGUMENT for null pointers, B, k or K < 1, k > K or
 *         K > INT32_MAX; UNSUPPORTED for B > INT32_MAX.
 */
rmm_status_t rmm_check_indices(const int32_t *idx, int64_t B, int64_t k, int64_t K, int32_t *bad,
                               hipStream_t stream);

/*
 * Gathered reduced product   (Sec. 3.2: RMM = A[:, I] B[I, :]; Sec. 3.3
 * projections Y~ = X[:, I] W[I, :]).
 *
 *   Y[b][m][n] = sum_{t < k} X[b][m][idx[b*k + t]] * W[idx[b*k + t]][n]
 *
 * X   : [B][M][ldx], ldx >= K.     W : [K][ldw], ldw >= N, shared by all units
 *       (row j of W is contraction index j; an nn.Linear weight [N][K] must
 *       be transposed once at load time).
 * idx : int32 [B*k], each unit's list strictly ascending with values in
 *       [0, K) -- e.g. from rmm_select, or any caller-chosen list (a static
 *       or random baseline).  Lists violating this are not detected; values
 *       outside [0, K) are undefined behaviour.
 * Y   : [B][M][ldy], ldy >= N, written (bf16 or fp32 per dtype).
 * The operands are gathered on the fly inside the GEMM; no compacted copy
 * of X[:, I] or W[I, :] is written to memory.
 * Errors: INVALID_ARGUMENT for null pointers, sizes < 1, k outside [1, K],
 *         ld too small, sizes above INT32_MAX.
 */
rmm_status_t rmm_reduced_gemm(const void *X, const void *W, const int32_t *idx,
                              rmm_dtype_t dtype, int64_t B, int64_t M, int64_t N,
                              int64_t K, int64_t k, int64_t ldx, int64_t ldw,
                              void *Y, int64_t ldy, hipStream_t stream);

/*
 * Reduced product for a decode step   (Sec. 3.2 definition of RMM; App. A:
 * during decoding the retained set follows the current decoding state).
 *
 * The same Y as rmm_reduced_gemm, for M <= 8 rows per unit (one token per
 * sequence in a decode step, or a few): reading the k retained rows of W is
 * the whole cost, and each is one contiguous row of W, so only those rows
 * are streamed from memory (k*N*2 bytes per unit).
 *
 * X, W, idx, Y, sizes : as rmm_reduced_gemm (bf16 only, M in [1, 8]).
 * workspace : rmm_gemv_workspace_size(B, M, N, k) bytes (0 is possible),
 *             16-byte aligned, or NULL when that size is 0; receives fp32
 *             partial sums when the retained list is split across
 *             workgroups, which a second kernel adds in a fixed order.
 * Errors    : as rmm_reduced_gemm; UNSUPPORTED for fp32, M > 8 or
 *             K*ldw*2 >= 2^31; WORKSPACE_TOO_SMALL.
 */
size_t rmm_gemv_workspace_size(int64_t B, int64_t M, int64_t N, int64_t k);
rmm_status_t rmm_reduced_gemv(const void *X, const void *W, const int32_t *idx,
                              rmm_dtype_t dtype, int64_t B, int64_t M, int64_t N,
                              int64_t K, int64_t k, int64_t ldx, int64_t ldw,
                              void *Y, int64_t ldy, void *workspace,
                              size_t workspace_bytes, hipStream_t stream);

/*
 * Gathered reduced product from K-major activations   (Sec. 3.2 definition
 * of RMM; Sec. 3.3 projections) -- the same Y as rmm_reduced_gemm, reading
 * X[:, I] as rows I of Xt (the copy written by rmm_score_kmajor).
 *
 *   Y[b][m][n] = sum_{t < k} Xt[b][idx[b*k + t]][m] * W[idx[b*k + t]][n]
 *
 * Xt  : [B][K][ldxt] bf16, ldxt >= M.     W : [K][ldw] bf16, ldw >= N.
 * idx : int32 [B*k], ascending per unit, values in [0, K).
 * Y   : [B][M][ldy] bf16, ldy >= N, written.
 * Retained rows of Xt and W are read as 16-byte vectors and staged through
 * LDS; no compacted operand is written to memory.  bf16 only.
 * Errors: INVALID_ARGUMENT for null pointers, sizes < 1, k outside [1, K],
 *         ld too small; UNSUPPORTED for Xt/W not 16-byte aligned, ldxt or ldw
 *         not multiples of 8, or K*ldxt or K*ldw of 2^30 elements or more.
 */
rmm_status_t rmm_reduced_gemm_kmajor(const void *Xt, const void *W, const int32_t *idx,
                                     int64_t B, int64_t M, int64_t N, int64_t K, int64_t k,
                                     int64_t ldxt, int64_t ldw, void *Y, int64_t ldy,
                                     hipStream_t stream);

/*
 * Reduced attention scores over head-dim slices   (Sec. 3.3, Attention:
 * S~ = (1/sqrt(d_h)) Q[:, I] K[:, I]^T, then the optional causal mask M).
 *
 *   S[b][h][i][t] = scale * sum_{u < k} Q[b][h][i][I(u)] * Kc[b][g][t][I(u)]
 *   with I = idx[(b*H + h)*k ..], g = h / (H / Hkv)  (consecutive query heads
 *   share a kv head), and S = -inf where causal != 0 and t > i + (Lk - Lq).
 *
 * Q     : [batch][H][Lq][D].   Kc : [batch][Hkv][Lk][D].
 * idx   : int32 [batch*H*k], ascending per head, values in [0, D) -- the
 *         per-head selection on Q (rmm_score + rmm_select with B = batch*H).
 * scale : multiplies the fp32 accumulator; the paper uses 1/sqrt(D) with
 *         the full head dimension.
 * S     : [batch][H][Lq][Lk], written in full (masked entries are -inf).
 * Errors: INVALID_ARGUMENT for null pointers, sizes < 1, H % Hkv != 0,
 *         k outside [1, D]; UNSUPPORTED for D > 256.
 */
rmm_status_t rmm_reduced_qk(const void *Q, const void *Kc, const int32_t *idx,
                            rmm_dtype_t dtype, int64_t batch, int64_t H,
                            int64_t Hkv, int64_t Lq, int64_t Lk, int64_t D,
                            int64_t k, float scale, int causal, void *S,
                            hipStream_t stream);

/*
 * Reduced attention scores with their softmax row statistics   (Sec. 3.3,
 * Attention: the reduced scores feed softmax(S~ + M); the Limitations
 * section names the memory movement of separate passes as a cost to remove).
 *
 * S exactly as rmm_reduced_qk writes it (bf16), and for each query row i of
 * each unit u = b*H + h:
 *   row_max[u*Lq + i]  = max over kept t of S[u][i][t]   (kept: not -inf)
 *   row_rinv[u*Lq + i] = 1 / sum over kept t of exp(S[u][i][t] - row_max)
 * in fp32 over the stored bf16 scores, summed in a fixed order; 0 and 0 for
 * a row with nothing kept (only when causal and Lq > Lk).  These are the
 * statistics rmm_attention_weights_kmajor computes in a pass of its own over
 * S; rmm_attention_weights_kmajor_rowstats takes them instead.
 * Q, Kc, idx, scale, causal as rmm_reduced_qk; bf16 only.
 * row_max, row_rinv : float [batch*H*Lq], 4-byte aligned, written.
 * Errors: INVALID_ARGUMENT as rmm_reduced_qk or for null statistics;
 *         UNSUPPORTED unless D is 64 or 128, Lk % 8 == 0, Lk <= 2^22, S is
 *         16-byte aligned and batch*H <= 65535.
 */
rmm_status_t rmm_reduced_qk_rowstats(const void *Q, const void *Kc, const int32_t *idx, int64_t batch,
                                     int64_t H, int64_t Hkv, int64_t Lq, int64_t Lk, int64_t D,
                                     int64_t k, float scale, int causal, void *S, float *row_max,
                                     float *row_rinv, hipStream_t stream);

/*
 * Reduced attention block   (Sec. 3.3 "Attention": the reduced scores feed
 * the softmax of the attention block, which then weights the value rows).
 *
 * O[b,h,i,:] = sum_t P[i,t] V[b,g,t,:],  P[i,:] = softmax(S[b,h,i,:] + M[i,:]),
 * with S the reduced scores of rmm_reduced_qk (same idx, scale, GQA map
 * g = h / (H / Hkv) and causal mask); S is never written to memory.  A query
 * row whose keys are all masked (only when Lq > Lk) gets O = 0.
 *
 * Q   : [batch][H][Lq][D]    Kc, V : [batch][Hkv][Lk][D]    O : [batch][H][Lq][D]
 *       (contiguous; the value rows have the head dimension D).
 * idx : int32 [batch*H*k], each head's list ascending (from rmm_select).
 * workspace : rmm_workspace_size(RMM_OP_ATTENTION, batch*H, Lk, D, k) bytes,
 *       16-byte aligned; receives each query head's retained key dims as
 *       contiguous rows (overwritten by every call).
 * Scores and the softmax are computed in fp32, the weights rounded to bf16
 * for the value product, fp32 accumulation, bf16 output.
 * Errors: INVALID_ARGUMENT as rmm_reduced_qk, or a misaligned workspace;
 *         UNSUPPORTED unless dtype is RMM_BF16, D == 128 and Q, Kc, V, O
 *         are 16-byte aligned; WORKSPACE_TOO_SMALL.
 */
rmm_status_t rmm_reduced_attention(const void *Q, const void *Kc, const void *V,
                                   const int32_t *idx, rmm_dtype_t dtype, int64_t batch,
                                   int64_t H, int64_t Hkv, int64_t Lq, int64_t Lk,
                                   int64_t D, int64_t k, float scale, int causal, void *O,
                                   void *workspace, size_t workspace_bytes,
                                   hipStream_t stream);

/*
 * Reduced gate|up projection feeding the reduced down projection   (Sec. 3.3
 * "MLP and linear projections": gate, up and down are each reduced, the down
 * projection selecting from its own input; that input is the MLP's
 * activation of the gate and up outputs, here SwiGLU as in the LLaMA-family
 * models the paper evaluates; the Limitations section names the memory
 * movement of separate scoring as a cost to remove).
 *
 * The gathered GEMM of rmm_reduced_gemm_kmajor over the gate and up weights,
 * whose epilogue applies the activation and writes the down projection's
 * K-major input and its column energies instead of the two outputs:
 *   g = bf16(X[:, I] Wg[I, :]),  u = bf16(X[:, I] Wu[I, :])   (as Y would be),
 *   Ht[b][c][m] = bf16(bf16(silu(g[m][c])) * u[m][c]),  silu(x) = x/(1+e^-x)
 *                 in fp32,
 *   energy[b][c] = sum over m < M of Ht[b][c][m]^2 (float64 sums of exact
 *                 squares, in a fixed order).
 * Feed them to rmm_select (K = F) and rmm_reduced_gemm_kmajor (Xt = Ht).
 *
 * Xt  : the MLP input's K-major copy [B][K][ldxt] (from rmm_score_kmajor).
 * Wgu : bf16 [K][ldw], 2F columns in 128-column blocks: block 2q holds the
 *       gate weights of channels 128q .. 128q+127, block 2q+1 the up weights
 *       of the same channels (a column permutation of [Wg | Wu] made once at
 *       load time).  idx: int32 [B*k] ascending, as for rmm_reduced_gemm.
 * Ht  : bf16 [B][F][ldht], ldht >= M, 16-byte aligned; columns M..ldht-1
 *       are not written.  energy: float64 [B][F], 8-byte aligned.
 * workspace : rmm_gemm_swiglu_workspace_size(B, M, F) bytes, 8-byte aligned
 *       (per-row-tile partial energies; overwritten by every call).
 * Errors : INVALID_ARGUMENT for null pointers, sizes < 1, k outside [1, K],
 *       ldxt < M, ldw < 2F or ldht < M; UNSUPPORTED unless F % 128 == 0,
 *       M % 8 == 0, ldht % 8 == 0, Ht 16-byte aligned and the conditions of
 *       rmm_reduced_gemm_kmajor hold; WORKSPACE_TOO_SMALL.
 */
size_t rmm_gemm_swiglu_workspace_size(int64_t B, int64_t M, int64_t F);
rmm_status_t rmm_reduced_gemm_swiglu_kmajor(const void *Xt, const void *Wgu, const int32_t *idx,
                                            int64_t B, int64_t M, int64_t F, int64_t K, int64_t k,
                                            int64_t ldxt, int64_t ldw, void *Ht, int64_t ldht,
                                            double *energy, void *workspace,
                                            size_t workspace_bytes, hipStream_t stream);

/*
 * Reduced attention block feeding a reduced projection   (Sec. 3.3: the
 * block's output is the input of the attention output projection, whose
 * retained set Sec. 3.2 scores from that input's columns; the Limitations
 * section names the memory movement of separate scoring as a cost to remove).
 *
 * The same block as rmm_reduced_attention (same arguments, same output
 * values bit for bit), written as the output projection's K-major input
 * instead of O, together with that input's column energies, so that the
 * projection needs no separate scoring pass:
 *   Ot[b][h*D + j][t] = O[b][h][t][j]        (heads concatenated along the
 *                                             projection's contraction axis)
 *   energy[b][h*D + j] = sum over t < Lq of Ot[b][h*D + j][t]^2
 * (float64 sums of the exact squares of the bf16 outputs, in a fixed order).
 * Feed them to rmm_select (B = batch, K = H*D) and rmm_reduced_gemm_kmajor
 * (Xt = Ot, ldxt = ldot, M = Lq).
 *
 * Ot     : bf16 [batch][H*D][ldot], ldot >= Lq, 16-byte aligned; columns
 *          Lq..ldot-1 are not written.
 * energy : float64 [batch][H*D], 8-byte aligned.
 * workspace : rmm_attention_kmajor_workspace_size(batch, H, Lq, Lk, D, k)
 *          bytes, 256-byte aligned (compacted key rows and per-query-tile
 *          partial energies; overwritten by every call).
 * Errors : as rmm_reduced_attention, plus INVALID_ARGUMENT for a null energy
 *          or ldot < Lq; UNSUPPORTED when Lq or ldot is not a multiple of 8
 *          or Ot is not 16-byte aligned.
 */
size_t rmm_attention_kmajor_workspace_size(int64_t batch, int64_t H, int64_t Lq, int64_t Lk,
                                            int64_t D, int64_t k);
rmm_status_t rmm_reduced_attention_kmajor(const void *Q, const void *Kc, const void *V,
                                          const int32_t *idx, rmm_dtype_t dtype, int64_t batch,
                                          int64_t H, int64_t Hkv, int64_t Lq, int64_t Lk,
                                          int64_t D, int64_t k, float scale, int causal, void *Ot,
                                          int64_t ldot, double *energy, void *workspace,
                                          size_t workspace_bytes, hipStream_t stream);

/*
 * Fused RMM projection   (Sec. 3.2 + Sec. 3.3 "MLP and linear projections").
 *
 * k = rmm_retained_count(r, K); then score -> rmm_select -> gathered GEMM
 * on `stream`, with no host synchronisation (k depends only on r and K).
 * Each of the B units selects from its own M rows.  For bf16 with 16-byte
 * aligned X rows and W (ldx, ldw multiples of 8) the K-major path is taken
 * (rmm_score_kmajor with the copy in the workspace, then
 * rmm_reduced_gemm_kmajor); otherwise rmm_score + rmm_reduced_gemm.
 *
 * idx_out   : int32 [B*k] receiving the index sets, or NULL (kept in the
 *             workspace).
 * workspace : rmm_workspace_size(RMM_OP_LINEAR, B, M, K, k) bytes, 256-byte
 *             aligned.  Other arguments as in rmm_reduced_gemm.
 * Errors    : as rmm_score / rmm_reduced_gemm, plus INVALID_ARGUMENT when
 *             r is not in (0, 1].
 */
rmm_status_t rmm_linear(const void *X, const void *W, double r, rmm_dtype_t dtype,
                        int64_t B, int64_t M, int64_t N, int64_t K, int64_t ldx,
                        int64_t ldw, void *Y, int64_t ldy, int32_t *idx_out,
                        void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Token-axis reduced value product   (Sec. 3.3, attention: token scores are
 * the column norms of the attention weights P, the value product keeps the
 * top ceil(rho_t * Lk) tokens; App. D: its MACs scale with rho_t).
 *
 *   a[u][t]    = sum_q P[u][q][t]^2             float64 (orders like the norm)
 *   T_u        = TopK(a[u], kt)                  ties -> lower index, ascending
 *   O[u][q][d] = sum_{t in T_u} P[u][q][t] * V[v(u)][t][d]
 *
 * with u = b*H + h over the batch*H query heads and v(u) = b*Hkv + h/(H/Hkv)
 * their shared value head.  Run as rmm_score over each head's Lq rows, one
 * rmm_select per head, then one gathered product per (sequence, kv head)
 * with that head's H/Hkv query heads as units (K-major path as rmm_linear).
 *
 * P   : [batch][H][Lq][ldp] (e.g. softmax probabilities), ldp >= Lk.
 * V   : [batch][Hkv][Lk][D], rows contiguous.  Same dtype as P.
 * O   : [batch][H][Lq][D], written.
 * kt  : tokens kept per head, 1 <= kt <= Lk (rmm_retained_count(rho_t, Lk)).
 * idx_out   : int32 [batch*H*kt] receiving the token sets, or NULL (kept in
 *             the workspace).
 * workspace : rmm_workspace_size(RMM_OP_PV, batch*H, Lq, Lk, kt) bytes,
 *             256-byte aligned.
 * Errors    : INVALID_ARGUMENT for null P/V/O, sizes < 1, H % Hkv != 0, kt
 *             outside [1, Lk], ldp < Lk, or a misaligned workspace;
 *             UNSUPPORTED when batch*H exceeds the grid limit;
 *             WORKSPACE_TOO_SMALL.
 */
rmm_status_t rmm_reduced_pv(const void *P, const void *V, rmm_dtype_t dtype, int64_t batch,
                            int64_t H, int64_t Hkv, int64_t Lq, int64_t Lk, int64_t D,
                            int64_t ldp, int64_t kt, void *O, int32_t *idx_out,
                            void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * rmm_linear without a caller workspace, for callers that cannot allocate
 * device memory: code under HIP graph capture, serving loops, harnesses that
 * forbid hipMalloc.
 *
 * Computes exactly what rmm_linear computes (the same kernels in the same
 * order: bit-identical Y and index sets), with the workspace taken from a
 * fixed device array inside the library instead of the caller's buffer.
 * That array holds rmm_noalloc_scratch_bytes() = 64 MiB on every GPU the
 * library runs on, from the first call on that GPU until the process ends;
 * the call itself allocates nothing (no hipMalloc, no hipFree, no library
 * routine that allocates).  rmm_workspace_size(RMM_OP_LINEAR, B, M, K, k)
 * must not exceed it (e.g. M*K up to about 30 million bf16 activations for
 * one unit).  Nothing in the array needs to start at zero: every byte a
 * call reads was written earlier in the same call.
 *
 * Every call on one GPU uses that GPU's one array, so calls that overlap in
 * time on one GPU (concurrent streams, or host threads) race and give
 * undefined results; serialise them (one stream, or events).  `stream` must
 * belong to the current device (NULL = its legacy default stream).
 *
 * Arguments as rmm_linear, without the workspace.
 * Errors: as rmm_linear; RMM_ERR_TOO_LARGE (before any HIP call) when the
 *         workspace rmm_linear would need exceeds the array;
 *         INVALID_ARGUMENT when `stream` belongs to another device.
 */
size_t rmm_noalloc_scratch_bytes(void);
rmm_status_t rmm_linear_noalloc(const void *X, const void *W, double r, rmm_dtype_t dtype,
                                int64_t B, int64_t M, int64_t N, int64_t K, int64_t ldx,
                                int64_t ldw, void *Y, int64_t ldy, int32_t *idx_out,
                                hipStream_t stream);

/*
 * Attention weights written K-major with their token energies   (Sec. 3.3,
 * attention: the token-axis reduction of the value product ranks tokens by
 * the column norms of the attention weights P = softmax(S + M); the
 * Limitations section names the memory movement of a separate scoring pass
 * as a cost to remove).
 *
 * For every unit u = b*H + h (query head) and query row i:
 *   kept(i, t)   = S[u][i][t] > -inf, and t <= i + (Lk - Lq) when causal
 *   rmax_i       = max over kept t of S[u][i][t],   rsum_i = sum over kept t
 *                  of exp(S[u][i][t] - rmax_i)                          (fp32)
 *   Pt[u][t][i]  = bf16(exp(S[u][i][t] - rmax_i) / rsum_i) where kept, else 0
 *                  (a row with nothing kept is all zero); with the causal
 *                  mask the zeros above the diagonal are written only where
 *                  i >= 256 * floor((t - (Lk - Lq)) / 256), the 256-query
 *                  block holding column t's diagonal (what
 *                  rmm_reduced_pv_kmajor reads); Pt[u][t][i] for smaller i
 *                  is left as it was
 *   energy[u][t] = sum over i < Lq of Pt[u][t][i]^2    (float64 sums of exact
 *                  squares in a fixed order; orders tokens like ||P[:, t]||)
 * With the causal mask the masked scores are never read.  Feed the energies
 * to rmm_select (B = batch*H, K = Lk) and the sets to rmm_reduced_pv_kmajor.
 *
 * S     : bf16 [batch][H][Lq][lds], lds >= Lk (e.g. rmm_reduced_qk's output).
 * Pt    : bf16 [batch][H][Lk][ldpt], ldpt >= Lq; columns Lq.. are not written.
 * energy: float64 [batch*H*Lk].
 * workspace : rmm_attention_weights_kmajor_workspace_size(batch, H, Lq, Lk)
 *         bytes, 256-byte aligned (row statistics and partial energies).
 * Errors: INVALID_ARGUMENT for null pointers, sizes < 1, lds < Lk, ldpt < Lq,
 *         a misaligned workspace; UNSUPPORTED unless S and Pt are 16-byte
 *         aligned, lds and ldpt are multiples of 8 and batch*H <= 65535;
 *         WORKSPACE_TOO_SMALL.
 */
size_t rmm_attention_weights_kmajor_workspace_size(int64_t batch, int64_t H, int64_t Lq, int64_t Lk);
rmm_status_t rmm_attention_weights_kmajor(const void *S, int64_t batch, int64_t H, int64_t Lq,
                                          int64_t Lk, int64_t lds, int causal, void *Pt,
                                          int64_t ldpt, double *energy, void *workspace,
                                          size_t workspace_bytes, hipStream_t stream);

/*
 * The same weights and energies from row statistics computed by the
 * producer of S   (Sec. 3.3, attention; the Limitations section's memory
 * movement of separate passes): rmax_i and rsum_i of
 * rmm_attention_weights_kmajor are replaced by the caller's
 *   Pt[u][t][i] = bf16(exp(S[u][i][t] - row_max[u*Lq + i]) * row_rinv[u*Lq + i])
 * where kept (zeros and energies as there), so that S is read once, by the
 * weights pass only.  With the statistics of rmm_reduced_qk_rowstats for
 * the same S the result agrees with rmm_attention_weights_kmajor up to the
 * order of the fp32 exponential sum.
 * row_max, row_rinv : float [batch*H*Lq], 4-byte aligned, read.
 * Other arguments, workspace and errors as rmm_attention_weights_kmajor
 * (the same workspace size), plus INVALID_ARGUMENT for null statistics and
 * UNSUPPORTED for misaligned ones.
 */
rmm_status_t rmm_attention_weights_kmajor_rowstats(const void *S, int64_t batch, int64_t H, int64_t Lq,
                                                   int64_t Lk, int64_t lds, int causal,
                                                   const float *row_max, const float *row_rinv,
                                                   void *Pt, int64_t ldpt, double *energy,
                                                   void *workspace, size_t workspace_bytes,
                                                   hipStream_t stream);

/*
 * Token-axis reduced value product from K-major weights   (Sec. 3.3: O =
 * P[:, T] V[T, :] with the kept tokens T of each query head; App. D: its
 * MACs scale with rho_t).
 *
 *   O[u][i][d] = sum over t in T_u of Pt[u][t][i] * V[v(u)][t][d]
 *
 * with T_u = idx[u*kt .. u*kt + kt) (ascending, from rmm_select on the
 * energies of rmm_attention_weights_kmajor) and v(u) = b*Hkv + h/(H/Hkv).
 * With causal != 0 the caller states that Pt[u][t][i] = 0 for t > i + (Lk -
 * Lq) (true of rmm_attention_weights_kmajor's causal output); the products
 * of those zeros are then skipped, whole 256-query tiles at a time.
 *
 * Pt : bf16 [batch][H][Lk][ldpt], ldpt >= Lq.   V : bf16 [batch][Hkv][Lk][D].
 * O  : bf16 [batch][H][Lq][D], written.
 * Errors: INVALID_ARGUMENT for null pointers, sizes < 1, H % Hkv != 0, kt
 *         outside [1, Lk], ldpt < Lq; UNSUPPORTED unless Pt and V are 16-byte
 *         aligned, ldpt and D are multiples of 8, Lk*ldpt*2 and Lk*D*2 are
 *         below 2^31 and batch*H <= 65535.
 */
rmm_status_t rmm_reduced_pv_kmajor(const void *Pt, const void *V, const int32_t *idx, int64_t batch,
                                   int64_t H, int64_t Hkv, int64_t Lq, int64_t Lk, int64_t D,
                                   int64_t kt, int64_t ldpt, int causal, void *O, hipStream_t stream);

/*
 * A decode step's reduced products, several at once   (Sec. 3.2 TopK of the
 * column norms and the reduced product; App. A: in decoding the retained
 * set follows the current token).
 *
 * For each group g and sequence b (one token per sequence), exactly what
 * rmm_select_tokens followed by rmm_reduced_gemv (M = 1) compute:
 *   idx_g[b] = TopK over j < K_g of X_g[b][j]^2   (ascending; ties to the
 *              lower index, NaN above +inf above every finite value)
 *   Y_g[b][n] = sum over t of X_g[b][idx_g[b][t]] * W_g[idx_g[b][t]][n]
 * in three launches for all groups together (selection, products, the
 * fixed-order reduction of split lists) instead of three per group (a group
 * of more than 32768 channels takes one more selection launch of its own).  The
 * groups must be independent of each other (no group reads another's Y);
 * within a model's layer step those are products whose inputs are ready
 * together.
 *
 * groups   : host array of ngroups (1..8) descriptions; per group X bf16
 *            [B][ldx] (16-byte aligned, ldx % 8 == 0, ldx >= K),
 *            W bf16 [K][ldw] (16-byte aligned, ldw % 8 == 0, ldw >= N),
 *            idx int32 [B][k] written, Y bf16 [B][ldy] written, 1 <= k <= K.
 * workspace: rmm_decode_step_workspace_size(groups, ngroups, B) bytes,
 *            256-byte aligned, or NULL when that is 0 (fp32 partial sums).
 * Errors   : INVALID_ARGUMENT for null pointers, sizes < 1, k outside
 *            [1, K], ld too small, a misaligned workspace; UNSUPPORTED for
 *            more than 8 groups, B > 65535, misaligned X or W,
 *            ldx or ldw not multiples of 8, K*ldw*2 >= 2^31;
 *            WORKSPACE_TOO_SMALL.
 */
typedef struct rmm_decode_group {
    const void *X;
    const void *W;
    int32_t *idx;
    void *Y;
    int64_t K, N, k, ldx, ldw, ldy;
} rmm_decode_group_t;
size_t rmm_decode_step_workspace_size(const rmm_decode_group_t *groups, int ngroups, int64_t B);
rmm_status_t rmm_decode_step(const rmm_decode_group_t *groups, int ngroups, int64_t B,
                             void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * The reduced products of a decode step over caller-made sets, several at
 * once   (Sec. 3.2 reduced product; the boundary accepts any ascending list,
 * e.g. sets computed for an earlier token or by another call).
 *
 * For each group g and sequence b: Y_g[b][n] = sum over t of
 * X_g[b][idx_g[b][t]] * W_g[idx_g[b][t]][n], exactly what rmm_reduced_gemv
 * (M = 1) computes, in two launches for all groups together (the products,
 * then the fixed-order reduction of split lists): rmm_decode_step without
 * its selection.  idx_g is read, not written: int32 [B][k], each list
 * strictly ascending within [0, K) (not checked on the device; an index
 * outside it reads outside W).
 *
 * groups, workspace, errors: as rmm_decode_step (the same workspace size).
 */
rmm_status_t rmm_decode_products(const rmm_decode_group_t *groups, int ngroups, int64_t B,
                                 void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * The reduced products of a decode step for a batch of sequences, each
 * weight row read once for the whole batch   (Sec. 3.2 reduced product; App.
 * A: each sequence's set follows its own current token).
 *
 * For each group g and sequence b < B: Y_g[b][n] = sum over t of
 * X_g[b][idx_g[b][t]] * W_g[idx_g[b][t]][n] -- what rmm_decode_products
 * computes -- but instead of reading k rows of W for every sequence
 * (B*k*N*2 bytes), the rows of the union of the B sets are streamed once and
 * multiplied by all sequences together on the matrix cores, each sequence
 * taking exact zeros for the rows it does not keep.  Worth it once B*r
 * exceeds about 1 (the per-sequence reads then exceed the whole of W).
 * Results equal rmm_decode_products' within rounding (another order of the
 * additions), not bit for bit.  W must be finite in the union's rows: a
 * sequence's zero times an infinite or NaN weight of a row that only other
 * sequences keep would make its output NaN.
 *
 * groups   : as rmm_decode_products (idx_g read: int32 [B][k], each list
 *            strictly ascending within [0, K); a list that is not gives
 *            undefined values but no access outside the buffers).
 * B        : 1..32 sequences.
 * workspace: rmm_decode_products_shared_workspace_size(groups, ngroups, B)
 *            bytes (never 0), 256-byte aligned.
 * Four launches for all groups together: the range boundaries of each list,
 * the union of every 512-index range with the activations over it, the
 * products (fp32 partials per range), the fixed-order reduction of the
 * ranges.
 * Errors   : as rmm_decode_products; UNSUPPORTED also for B > 32.
 */
size_t rmm_decode_products_shared_workspace_size(const rmm_decode_group_t *groups, int ngroups,
                                                 int64_t B);
rmm_status_t rmm_decode_products_shared(const rmm_decode_group_t *groups, int ngroups, int64_t B,
                                        void *workspace, size_t workspace_bytes,
                                        hipStream_t stream);

/*
 * A decode step for a batch of sequences   (App. A: each sequence's set
 * follows its own current token; Sec. 3.2 reduced product): for each group,
 * idx_g[b] = the TopK of X_g[b]^2 as rmm_decode_step selects it (the same
 * lists, bit for bit), then Y_g = rmm_decode_products_shared's products over
 * them -- one selection launch for all groups (plus one per group wider than
 * 32768 channels) and the four launches of the shared products.
 *
 * groups, B, workspace, errors: as rmm_decode_products_shared (the same
 * workspace size); idx_g is written.
 */
rmm_status_t rmm_decode_step_shared(const rmm_decode_group_t *groups, int ngroups, int64_t B,
                                    void *workspace, size_t workspace_bytes, hipStream_t stream);

/* Static, NUL-terminated description of a status code (never NULL). */
const char *rmm_status_string(rmm_status_t status);

#ifdef __cplusplus
}
#endif

#endif /* RMM_H */
