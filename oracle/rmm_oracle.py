"""CPU oracle for Reduced Matrix Multiplication (RMM) -- TEST INFRASTRUCTURE.

This module is the plain, slow, obviously-correct statement of what the RMM
hot path computes.  It exists to check the HIP library against; it is not a
fallback and is never on the product path.  Only the test suite, the smoke
check of ``__graft_entry__`` and the CPU-baseline leg of ``bench.py`` may
import it.  It shares no code with the HIP path.

Everything is float64.  Inputs are the exact values of the stored bf16 or
fp32 tensors (see ``workloads.decode``); every square and every product of
two such values is exact in float64.

Paper passages followed (arXiv 2608.13426, "Reduced Matrix Multiplication"):

* Sec. 3.2, definition of RMM: for Y = AB with A in R^{n x d}, B in R^{d x m},
  pick I subset of [d] with |I| = ceil(rho * d), rho in (0, 1], and return
  A[:, I] B[I, :].
* Sec. 3.2, "Activation-aware dimension selection": score s_j = ||A[:, j]||_2,
  I = TopK(s, ceil(rho * d)).
* Sec. 3.3, "MLP and linear projections": the same rule with A = X, B = W.
* Sec. 3.3, "Attention": per head, scores on the columns of Q; the reduced
  scores are (1 / sqrt(d_h)) Q[:, I] K[:, I]^T with the full d_h in the
  scale; the optional causal mask M is added before the softmax; with
  grouped-query attention the selection is made per query head and applied
  to the shared K.  Optionally the value product PV is reduced over the
  token axis: token scores a_t = ||P[:, t]||_2, T = TopK(a, ceil(rho_t L_k)),
  O = P[:, T] V[T, :].
* Sec. 3.5 and Appendix E: the rank-one decomposition, the error bound
  (Proposition "RMM Approximation Error Bound"), the factorised bound
  (Corollary) and the normalised bound with the discarded-energy ratios;
  Appendix B.4 defines the retained-energy diagnostic.
* The MLP activation between the reduced gate/up and down projections of
  the evaluated LLaMA-family models: silu(gate) * up (used to chain the
  projections; it is the models' own operation, not part of RMM).
* The normalisation that produces the inputs of the attention and MLP
  projections in those models, RMSNorm (again the models' own operation,
  used to chain a producer into a reduced projection), and the attention
  weights softmax(S + M) whose column norms Sec. 3.3 ranks for the
  token-axis value product.
* Appendix A, "Inference setup": the index set is recomputed per affected
  product from the current sequence's activation block (one selection per
  sequence; one per query head on the attention side).

Readings where the paper is silent (each also listed in the design notes):

* k for a floating-point rho: ceil(rho*K) of the decimal the caller meant --
  if rho*K is within 1e-9*K of an integer, that integer is taken.
* Ranking uses the energies e_j = s_j^2 (sqrt is monotone).  e_j is the exact
  sum of the exact squares, rounded once to float64 (math.fsum).  The
  ranking decision is therefore taken in float64.
* Ties go to the lower index; a NaN energy ranks above +inf, which ranks
  above every finite energy; all NaNs tie with each other.
* The index set is returned in ascending order.
* GQA: query head h reads kv head h // (H / Hkv) (consecutive query heads
  share one kv head).
* Causal mask: entry (i, t) is masked iff t > i + (Lk - Lq) (bottom-right
  aligned); masked entries are -inf, so softmax(S + M) is softmax of S with
  those entries removed.
* Reduced attention block (softmax(S + M) V with the reduced S): a query row
  whose keys are all masked (only when Lq > Lk) has no weights; its output
  is 0.
"""
from __future__ import annotations

import math

import numpy as np

__all__ = [
    "retained_count", "column_energies", "topk_indices", "reduced_matmul",
    "rmm", "rmm_batched", "gqa_kv_head", "reduced_qk", "rmm_qk", "reduced_attention",
    "reduced_pv", "silu", "swiglu", "rmsnorm", "attention_weights", "softmax_row_stats",
    "residual_energy", "retained_energy_fraction", "discarded_energy_ratio",
    "rank_one_bound", "factorized_bound", "normalized_bound",
    "selection_margin",
]


# ---------------------------------------------------------------------------
# Sec. 3.2: |I| = ceil(rho * d)
# ---------------------------------------------------------------------------

def retained_count(r: float, K: int) -> int:
    """Number of retained indices, ceil(r*K), for r in (0, 1] (Sec. 3.2).

    Raises ValueError outside the domain (r <= 0, r > 1, NaN, K < 1).
    """
    if not isinstance(K, (int, np.integer)) or K < 1:
        raise ValueError("K must be a positive integer")
    r = float(r)
    if not (r > 0.0 and r <= 1.0):          # also rejects NaN
        raise ValueError("retention ratio must lie in (0, 1]")
    p = r * K
    nearest = round(p)
    if abs(p - nearest) <= 1e-9 * K:
        k = int(nearest)
    else:
        k = math.ceil(p)
    return max(1, min(int(K), k))


# ---------------------------------------------------------------------------
# Sec. 3.2: scores s_j = ||A[:, j]||_2, ranked through e_j = s_j^2
# ---------------------------------------------------------------------------

def column_energies(A: np.ndarray) -> np.ndarray:
    """e_j = sum_i A[i, j]^2 for A [n x d]; exact sum rounded once to float64.

    The squares are exact in float64 for bf16/fp32 inputs; math.fsum returns
    the correctly rounded value of their exact sum, independent of order.
    """
    A = np.asarray(A, dtype=np.float64)
    if A.ndim != 2:
        raise ValueError("A must be 2-D [n x d]")
    sq = A * A
    return np.array([math.fsum(sq[:, j]) for j in range(A.shape[1])],
                    dtype=np.float64)


def _rank_key(e: float, j: int):
    """Sort key: NaN first, then larger energy first, then lower index."""
    if math.isnan(e):
        return (0, 0.0, j)
    return (1, -e, j)


def topk_indices(e: np.ndarray, k: int) -> np.ndarray:
    """I = TopK(e, k) as ascending int64 indices (Sec. 3.2).

    Total order: energy descending, ties to the lower index, NaN largest.
    """
    e = np.asarray(e, dtype=np.float64)
    K = e.shape[0]
    if not (1 <= k <= K):
        raise ValueError("k must lie in [1, K]")
    order = sorted(range(K), key=lambda j: _rank_key(float(e[j]), j))
    return np.array(sorted(order[:k]), dtype=np.int64)


# ---------------------------------------------------------------------------
# Sec. 3.2 / 3.3: the reduced product
# ---------------------------------------------------------------------------

def reduced_matmul(A: np.ndarray, B: np.ndarray, idx: np.ndarray) -> np.ndarray:
    """RMM with a given index set: A[:, I] @ B[I, :] in float64 (Sec. 3.2)."""
    A = np.asarray(A, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64)
    idx = np.asarray(idx, dtype=np.int64)
    return A[:, idx] @ B[idx, :]


def rmm(A: np.ndarray, B: np.ndarray, r: float):
    """Full RMM of one selection unit (Sec. 3.2, Sec. 3.3 projections).

    Returns (Y, idx, e): the reduced product, the ascending index set and
    the column energies of A.
    """
    A = np.asarray(A, dtype=np.float64)
    k = retained_count(r, A.shape[1])
    e = column_energies(A)
    idx = topk_indices(e, k)
    return reduced_matmul(A, B, idx), idx, e


def rmm_batched(X: np.ndarray, W: np.ndarray, r: float):
    """RMM over a batch of sequences X [b x n x d] sharing W [d x m].

    Each sequence is its own selection unit (Appendix A, prefill).
    Returns (Y [b x n x m], idx [b x k], e [b x d]).
    """
    X = np.asarray(X, dtype=np.float64)
    outs = [rmm(X[b], W, r) for b in range(X.shape[0])]
    return (np.stack([o[0] for o in outs]), np.stack([o[1] for o in outs]),
            np.stack([o[2] for o in outs]))


# ---------------------------------------------------------------------------
# Sec. 3.3: reduced attention scores over head-dim slices
# ---------------------------------------------------------------------------

def gqa_kv_head(h: int, H: int, Hkv: int) -> int:
    """kv head read by query head h: h // (H / Hkv)."""
    if H % Hkv:
        raise ValueError("H must be a multiple of Hkv")
    return h // (H // Hkv)


def reduced_qk(Q: np.ndarray, K: np.ndarray, idx: np.ndarray,
               causal: bool, rows=None) -> np.ndarray:
    """S[h] = (1/sqrt(D)) Q[h][:, I_h] K[g(h)][:, I_h]^T, masked (Sec. 3.3).

    Q [H x Lq x D], K [Hkv x Lk x D], idx [H x k] -> S [H x Lq x Lk] float64
    with -inf at masked entries (t > i + Lk - Lq) when ``causal``.  With
    ``rows`` (query positions i), only those rows of S are computed.
    """
    Q = np.asarray(Q, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    H, Lq, D = Q.shape
    Hkv, Lk, _ = K.shape
    rows = np.arange(Lq) if rows is None else np.asarray(rows, dtype=np.int64)
    scale = 1.0 / math.sqrt(D)
    S = np.empty((H, rows.shape[0], Lk), dtype=np.float64)
    i = rows[:, None]
    t = np.arange(Lk)[None, :]
    for h in range(H):
        g = gqa_kv_head(h, H, Hkv)
        I = np.asarray(idx[h], dtype=np.int64)
        S[h] = scale * (Q[h][rows][:, I] @ K[g][:, I].T)
        if causal:
            S[h][t > i + (Lk - Lq)] = -np.inf
    return S


def rmm_qk(Q: np.ndarray, K: np.ndarray, r: float, causal: bool):
    """Per-head selection on Q, then reduced scores (Sec. 3.3).

    Returns (S, idx [H x k], e [H x D]).
    """
    Q = np.asarray(Q, dtype=np.float64)
    H, _, D = Q.shape
    k = retained_count(r, D)
    e = np.stack([column_energies(Q[h]) for h in range(H)])
    idx = np.stack([topk_indices(e[h], k) for h in range(H)])
    return reduced_qk(Q, K, idx, causal), idx, e


def reduced_attention(Q: np.ndarray, K: np.ndarray, V: np.ndarray, idx: np.ndarray,
                      causal: bool, rows=None) -> np.ndarray:
    """O[h] = softmax(S[h] + M) V[g(h)] with the reduced scores S (Sec. 3.3).

    The attention block the paper places RMM in: the reduced scores of
    ``reduced_qk`` (the mask's -inf entries drop out of the softmax), then
    each query row averages the value rows of its kv head with the softmax
    weights.  Q [H x Lq x D], K [Hkv x Lk x D], V [Hkv x Lk x Dv], idx [H x k]
    -> O [H x Lq x Dv] float64.  A query row with every key masked (only
    possible when Lq > Lk) has no weights; its output is 0.  With ``rows``,
    only those query rows are computed.
    """
    V = np.asarray(V, dtype=np.float64)
    H = np.asarray(Q).shape[0]
    Hkv = np.asarray(K).shape[0]
    S = reduced_qk(Q, K, idx, causal, rows)
    O = np.zeros((H, S.shape[1], V.shape[2]), dtype=np.float64)
    for h in range(H):
        g = gqa_kv_head(h, H, Hkv)
        for i in range(S.shape[1]):
            s = S[h, i]
            keep = s != -np.inf                      # masked entries are -inf
            if not keep.any():
                continue
            w = np.zeros_like(s)
            w[keep] = np.exp(s[keep] - s[keep].max())
            O[h, i] = (w / w.sum()) @ V[g]
    return O


def reduced_pv(P: np.ndarray, V: np.ndarray, kt: int):
    """Token-axis reduced value product (Sec. 3.3, attention).

    P [H x Lq x Lk] holds the attention weights of H query heads, V
    [Hkv x Lk x Dv] the value rows of their kv heads.  For each head h: the
    token scores are the column norms of P[h], ranked by their squares
    a_t^2 = column_energies(P[h]); T_h = TopK(a, kt); the output is
    P[h][:, T_h] @ V[g(h)][T_h, :].  Returns (O [H x Lq x Dv] float64,
    idx [H x kt]).
    """
    P = np.asarray(P, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    H, Hkv = P.shape[0], V.shape[0]
    idx = np.stack([topk_indices(column_energies(P[h]), kt) for h in range(H)])
    O = np.stack([reduced_matmul(P[h], V[gqa_kv_head(h, H, Hkv)], idx[h]) for h in range(H)])
    return O, idx


# ---------------------------------------------------------------------------
# The MLP between the reduced gate/up and down projections
# ---------------------------------------------------------------------------

def silu(x: np.ndarray) -> np.ndarray:
    """SiLU, x * sigmoid(x) = x / (1 + exp(-x)), in float64.

    The MLP of the LLaMA-family models the paper evaluates (Sec. 4 setup;
    Sec. 3.3 reduces its up, gate and down projections) feeds the down
    projection with silu(gate output) * up output."""
    x = np.asarray(x, dtype=np.float64)
    with np.errstate(over="ignore"):
        return x / (1.0 + np.exp(-x))


def swiglu(g: np.ndarray, u: np.ndarray) -> np.ndarray:
    """The down projection's input: silu(g) * u, elementwise, float64."""
    return silu(g) * np.asarray(u, dtype=np.float64)


# ---------------------------------------------------------------------------
# The producers of the reduced products' inputs
# ---------------------------------------------------------------------------

def rmsnorm(X: np.ndarray, gamma: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm of each row of X [n x d] with weight gamma [d], float64:
    y[i, j] = gamma[j] * X[i, j] / sqrt(mean_j X[i, j]^2 + eps).

    The normalisation in front of the attention and MLP projections of the
    LLaMA-family models the paper reduces (Sec. 4 setup, Sec. 3.3); its
    output is the activation block X whose column norms Sec. 3.2 ranks."""
    X = np.asarray(X, dtype=np.float64)
    gamma = np.asarray(gamma, dtype=np.float64)
    ms = np.array([math.fsum((X[i] * X[i]).tolist()) for i in range(X.shape[0])]) / X.shape[1]
    return X / np.sqrt(ms + float(eps))[:, None] * gamma[None, :]


def attention_weights(S: np.ndarray) -> np.ndarray:
    """P = softmax(S + M) over the last axis, float64 (Sec. 3.3: the
    attention weights whose column norms rank the tokens of the value
    product).  Masked entries are -inf in S and get weight 0; a row with
    every entry masked gets all zeros."""
    S = np.asarray(S, dtype=np.float64)
    P = np.zeros_like(S)
    flat_S, flat_P = S.reshape(-1, S.shape[-1]), P.reshape(-1, S.shape[-1])
    for i in range(flat_S.shape[0]):
        s = flat_S[i]
        keep = s != -np.inf
        if not keep.any():
            continue
        w = np.exp(s[keep] - s[keep].max())
        flat_P[i, keep] = w / math.fsum(w.tolist())
    return P


def softmax_row_stats(S: np.ndarray):
    """The two numbers per row that define softmax(S + M) over the last axis
    (Sec. 3.3, attention): the largest kept score m and the reciprocal of the
    sum over kept keys of exp(s - m), in float64, as (m, rinv) with the
    leading shape of S.  Masked entries are -inf and not kept; a row with
    every entry masked gets (0, 0)."""
    S = np.asarray(S, dtype=np.float64)
    flat = S.reshape(-1, S.shape[-1])
    m = np.zeros(flat.shape[0])
    rinv = np.zeros(flat.shape[0])
    for i in range(flat.shape[0]):
        s = flat[i]
        keep = s != -np.inf
        if not keep.any():
            continue
        m[i] = s[keep].max()
        rinv[i] = 1.0 / math.fsum(np.exp(s[keep] - m[i]).tolist())
    return m.reshape(S.shape[:-1]), rinv.reshape(S.shape[:-1])


# ---------------------------------------------------------------------------
# Sec. 3.5 / Appendix E: energies and error bounds
# ---------------------------------------------------------------------------

def _complement(idx: np.ndarray, d: int) -> np.ndarray:
    keep = np.zeros(d, dtype=bool)
    keep[np.asarray(idx, dtype=np.int64)] = True
    return np.nonzero(~keep)[0]


def residual_energy(e: np.ndarray, idx: np.ndarray) -> float:
    """sum_{j not in I} e_j, the quantity TopK minimises (Theorem, App. E)."""
    e = np.asarray(e, dtype=np.float64)
    return math.fsum(e[_complement(idx, e.shape[0])])


def retained_energy_fraction(e: np.ndarray, idx: np.ndarray) -> float:
    """Share of the activation squared norm kept by I (Appendix B.4)."""
    e = np.asarray(e, dtype=np.float64)
    total = math.fsum(e)
    return math.fsum(e[np.asarray(idx, dtype=np.int64)]) / total


def discarded_energy_ratio(A: np.ndarray, idx: np.ndarray, axis: int) -> float:
    """eps = ||A restricted to discarded slices||_F^2 / ||A||_F^2 (Sec. 3.5).

    axis=1: discarded columns (eps_A); axis=0: discarded rows (eps_B).
    """
    A = np.asarray(A, dtype=np.float64)
    comp = _complement(idx, A.shape[axis])
    part = A[:, comp] if axis == 1 else A[comp, :]
    return math.fsum((part * part).ravel()) / math.fsum((A * A).ravel())


def rank_one_bound(A: np.ndarray, B: np.ndarray, idx: np.ndarray) -> float:
    """sum_{j not in I} ||A[:, j]||_2 ||B[j, :]||_2 (Proposition, App. E)."""
    A = np.asarray(A, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64)
    comp = _complement(idx, A.shape[1])
    return math.fsum(float(np.linalg.norm(A[:, j]) * np.linalg.norm(B[j, :]))
                     for j in comp)


def factorized_bound(A: np.ndarray, B: np.ndarray, idx: np.ndarray) -> float:
    """||A[:, Ibar]||_F ||B[Ibar, :]||_F (Corollary, App. E)."""
    A = np.asarray(A, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64)
    comp = _complement(idx, A.shape[1])
    return float(np.linalg.norm(A[:, comp]) * np.linalg.norm(B[comp, :]))


def normalized_bound(A: np.ndarray, B: np.ndarray, idx: np.ndarray) -> float:
    """sqrt(eps_A * eps_B), the bound on the relative error (Sec. 3.5)."""
    return math.sqrt(discarded_energy_ratio(A, idx, 1) *
                     discarded_energy_ratio(B, idx, 0))


# ---------------------------------------------------------------------------
# float64 decision margin at the k boundary
# ---------------------------------------------------------------------------

def selection_margin(e: np.ndarray, k: int) -> float:
    """Relative gap between the k-th and (k+1)-th largest energies.

    Returns +inf when k == d (nothing is excluded) and 0 for an exact tie.
    A GPU sum of n squares in float64, in any order, is within about
    n * 2^-53 (relative) of the exact sum; if this margin is larger than
    twice that, every float64 summation order selects the same set.
    """
    e = np.asarray(e, dtype=np.float64)
    K = e.shape[0]
    if k >= K:
        return math.inf
    order = sorted(range(K), key=lambda j: _rank_key(float(e[j]), j))
    a, b = float(e[order[k - 1]]), float(e[order[k]])
    if math.isnan(a):
        return 0.0 if math.isnan(b) else math.inf
    if a == b:
        return 0.0
    if math.isinf(a):
        return math.inf
    return (a - b) / a
