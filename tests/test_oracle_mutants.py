"""The pins are strong enough: each planted mistake in the oracle fails one.

Mistakes are planted into the oracle module on the CPU (monkeypatch), never
into the HIP path.
"""
import math

import numpy as np
import pytest

from oracle import rmm_oracle as ro
from tests import pins

_reduced_qk = ro.reduced_qk          # unpatched, for mutants built on it


def _k_plain_ceil(r, K):
    if not (0 < r <= 1):
        raise ValueError
    return max(1, math.ceil(r * K))


def _k_round(r, K):
    if not (0 < r <= 1):
        raise ValueError
    return max(1, round(r * K))


def _k_no_domain(r, K):
    p = r * K
    n = round(p) if p == p and abs(p) != math.inf else 1
    return max(1, min(K, int(n) if abs(p - n) <= 1e-9 * K else math.ceil(p)))


def _e_l1(A):
    A = np.asarray(A, dtype=np.float64)
    return np.array([math.fsum(np.abs(A[:, j])) for j in range(A.shape[1])])


def _e_drop_row(A):
    A = np.asarray(A, dtype=np.float64)[1:]
    return np.array([math.fsum(A[:, j] ** 2) for j in range(A.shape[1])])


def _e_rows(A):
    A = np.asarray(A, dtype=np.float64)
    r = np.array([math.fsum(A[i, :] ** 2) for i in range(A.shape[0])])
    return np.resize(r, A.shape[1])


def _topk_smallest(e, k):
    order = sorted(range(len(e)), key=lambda j: (float(e[j]), j))
    return np.array(sorted(order[:k]))


def _topk_ties_high(e, k):
    order = sorted(range(len(e)), key=lambda j: (ro._rank_key(float(e[j]), 0), -j))
    return np.array(sorted(order[:k]))


def _topk_unsorted(e, k):
    order = sorted(range(len(e)), key=lambda j: ro._rank_key(float(e[j]), j))
    return np.array(order[:k])


def _topk_nan_low(e, k):
    order = sorted(range(len(e)),
                   key=lambda j: (1, 0.0, j) if math.isnan(e[j]) else (0, -float(e[j]), j))
    return np.array(sorted(order[:k]))


def _mm_transposed(A, B, idx):
    A = np.asarray(A, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64)
    if B.shape[0] == B.shape[1]:
        return A[:, idx] @ B[:, idx].T
    return A[:, idx] @ B[idx, :]


def _mm_off_by_one(A, B, idx):
    A = np.asarray(A, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64)
    idx = np.asarray(idx)
    return A[:, idx] @ B[np.minimum(idx + 1, B.shape[0] - 1), :]


def _mm_sign(A, B, idx):
    A = np.asarray(A, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64)
    out = A[:, idx] @ B[idx, :]
    out[:, -1] *= -1
    return out


def _qk_patch(body):
    def f(Q, K, idx, causal):
        Q = np.asarray(Q, dtype=np.float64)
        K = np.asarray(K, dtype=np.float64)
        H, Lq, D = Q.shape
        Hkv, Lk, _ = K.shape
        S = np.empty((H, Lq, Lk))
        for h in range(H):
            S[h] = body(Q, K, np.asarray(idx[h]), h, H, Hkv, D)
            if causal:
                i = np.arange(Lq)[:, None]
                t = np.arange(Lk)[None, :]
                S[h][t > i + (Lk - Lq)] = -np.inf
        return S
    return f


_qk_scale_k = _qk_patch(lambda Q, K, I, h, H, Hkv, D:
                        Q[h][:, I] @ K[h // (H // Hkv)][:, I].T / math.sqrt(len(I)))
_qk_gqa_mod = _qk_patch(lambda Q, K, I, h, H, Hkv, D:
                        Q[h][:, I] @ K[h % Hkv][:, I].T / math.sqrt(D))
_qk_no_scale = _qk_patch(lambda Q, K, I, h, H, Hkv, D:
                         Q[h][:, I] @ K[h // (H // Hkv)][:, I].T)


def _qk_mask_off_by_one(Q, K, idx, causal):
    S = _reduced_qk(Q, K, idx, False)
    if causal:
        Lq, Lk = S.shape[1], S.shape[2]
        i = np.arange(Lq)[:, None]
        t = np.arange(Lk)[None, :]
        for h in range(S.shape[0]):
            S[h][t >= i + (Lk - Lq)] = -np.inf
    return S


def _qk_mask_top_left(Q, K, idx, causal):
    S = _reduced_qk(Q, K, idx, False)
    if causal:
        Lq, Lk = S.shape[1], S.shape[2]
        i = np.arange(Lq)[:, None]
        t = np.arange(Lk)[None, :]
        for h in range(S.shape[0]):
            S[h][t > i] = -np.inf
    return S


def _rmm_qk_scores_k(Q, K, r, causal):
    Q = np.asarray(Q, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    H, _, D = Q.shape
    k = ro.retained_count(r, D)
    e = np.stack([ro.column_energies(K[h * K.shape[0] // H]) for h in range(H)])
    idx = np.stack([ro.topk_indices(e[h], k) for h in range(H)])
    return ro.reduced_qk(Q, K, idx, causal), idx, e


def _attn_patch(weights, value_head):
    """reduced_attention with the per-row weights or the value head replaced."""
    def f(Q, K, V, idx, causal, rows=None):
        V = np.asarray(V, dtype=np.float64)
        H, Hkv = np.asarray(Q).shape[0], np.asarray(K).shape[0]
        S = ro.reduced_qk(Q, K, idx, causal, rows)
        O = np.zeros((H, S.shape[1], V.shape[2]))
        for h in range(H):
            W = weights(S[h])
            O[h] = np.nan_to_num(W) @ V[value_head(h, H, Hkv)]
        return O
    return f


def _w_softmax(S):
    out = np.zeros_like(S)
    for i, s in enumerate(S):
        keep = s != -np.inf
        if keep.any():
            w = np.exp(s[keep] - s[keep].max())
            out[i, keep] = w / w.sum()
    return out


def _w_over_queries(S):
    E = np.where(S == -np.inf, 0.0, np.exp(np.where(S == -np.inf, 0.0, S)))
    return E / np.maximum(E.sum(axis=0, keepdims=True), 1e-300)


def _w_unnormalised(S):
    return np.where(S == -np.inf, 0.0, np.exp(np.where(S == -np.inf, 0.0, S)))


def _w_mask_as_zero(S):
    return _w_softmax(np.where(S == -np.inf, 0.0, S))


_gqa = lambda h, H, Hkv: h // (H // Hkv)
_attn_over_queries = _attn_patch(_w_over_queries, _gqa)
_attn_unnormalised = _attn_patch(_w_unnormalised, _gqa)
_attn_mask_as_zero = _attn_patch(_w_mask_as_zero, _gqa)
_attn_gqa_modulo = _attn_patch(_w_softmax, lambda h, H, Hkv: h % Hkv)


def _pv_patch(energies, value_head):
    """reduced_pv with the token scores or the value head replaced."""
    def f(P, V, kt):
        P, V = np.asarray(P, dtype=np.float64), np.asarray(V, dtype=np.float64)
        H, Hkv = P.shape[0], V.shape[0]
        idx = np.stack([ro.topk_indices(energies(P[h]), kt) for h in range(H)])
        O = np.stack([ro.reduced_matmul(P[h], V[value_head(h, H, Hkv)], idx[h]) for h in range(H)])
        return O, idx
    return f


_pv_scores_rows = _pv_patch(lambda A: ro.column_energies(A.T), _gqa)
_pv_scores_l1 = _pv_patch(lambda A: np.abs(A).sum(axis=0), _gqa)
_pv_gqa_modulo = _pv_patch(ro.column_energies, lambda h, H, Hkv: h % Hkv)


def _silu_sigmoid(x):
    x = np.asarray(x, dtype=np.float64)
    return 1.0 / (1.0 + np.exp(-x))


def _silu_sign(x):
    x = np.asarray(x, dtype=np.float64)
    return x / (1.0 + np.exp(x))


def _swiglu_swapped(g, u):
    return ro.silu(u) * np.asarray(g, dtype=np.float64)


def _rms_sum(X, gamma, eps):          # sum of squares instead of the mean
    X = np.asarray(X, dtype=np.float64)
    return X / np.sqrt((X * X).sum(axis=1) + eps)[:, None] * np.asarray(gamma, dtype=np.float64)


def _rms_eps_outside(X, gamma, eps):   # eps added after the square root
    X = np.asarray(X, dtype=np.float64)
    return X / (np.sqrt((X * X).mean(axis=1)) + eps)[:, None] * np.asarray(gamma, dtype=np.float64)


def _rms_gamma_rows(X, gamma, eps):    # weight applied along rows
    X = np.asarray(X, dtype=np.float64)
    y = X / np.sqrt((X * X).mean(axis=1) + eps)[:, None]
    g = np.asarray(gamma, dtype=np.float64)
    return y * np.resize(g, X.shape[0])[:, None]


def _rms_l1(X, gamma, eps):            # mean absolute value
    X = np.asarray(X, dtype=np.float64)
    return X / (np.abs(X).mean(axis=1) + eps)[:, None] * np.asarray(gamma, dtype=np.float64)


def _aw_over_queries(S):               # normalised over the query axis
    S = np.asarray(S, dtype=np.float64)
    return np.swapaxes(ro_attention_weights(np.swapaxes(S, -1, -2)), -1, -2)


def _aw_unnormalised(S):
    S = np.asarray(S, dtype=np.float64)
    m = np.max(np.where(np.isfinite(S), S, -1e300), axis=-1, keepdims=True)
    return np.where(np.isfinite(S), np.exp(S - m), 0.0)


def _aw_no_max(S):                     # no shift by the row max and no empty-row rule:
    S = np.asarray(S, dtype=np.float64)  # a fully masked row divides 0 by 0
    E = np.where(np.isfinite(S), np.exp(S), 0.0)
    with np.errstate(invalid="ignore"):
        return E / E.sum(axis=-1, keepdims=True)


def _rs_min(S):                        # the row minimum instead of the maximum
    S = np.asarray(S, dtype=np.float64)
    keep = np.isfinite(S)
    m = np.where(keep.any(axis=-1), np.min(np.where(keep, S, np.inf), axis=-1), 0.0)
    e = np.where(keep, np.exp(np.where(keep, S, 0.0) - m[..., None]), 0.0).sum(axis=-1)
    return m, np.where(e > 0, 1.0 / np.where(e > 0, e, 1.0), 0.0)


def _rs_sum_not_recip(S):              # the sum, not its reciprocal
    m, rinv = ro_softmax_row_stats(S)
    return m, np.where(rinv > 0, 1.0 / np.where(rinv > 0, rinv, 1.0), 0.0)


def _rs_over_first_axis(S):            # statistics over the first axis
    S = np.asarray(S, dtype=np.float64)
    m, rinv = ro_softmax_row_stats(np.moveaxis(S, 0, -1))
    return m.T if m.ndim == 2 else m, rinv.T if rinv.ndim == 2 else rinv


ro_attention_weights = ro.attention_weights
ro_softmax_row_stats = ro.softmax_row_stats

def _b1_kept(A, B, idx):
    # sums over the kept indices instead of the discarded ones
    A = np.asarray(A, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64)
    return math.fsum(float(np.linalg.norm(A[:, j]) * np.linalg.norm(B[j, :]))
                     for j in np.asarray(idx, dtype=np.int64))


def _b2_whole_b(A, B, idx):
    # the factorized bound with all of B's rows
    A = np.asarray(A, dtype=np.float64)
    comp = ro._complement(idx, A.shape[1])
    return float(np.linalg.norm(A[:, comp]) * np.linalg.norm(np.asarray(B, dtype=np.float64)))


def _bn_no_sqrt(A, B, idx):
    return ro.discarded_energy_ratio(A, idx, 1) * ro.discarded_energy_ratio(B, idx, 0)


MUTANTS = {
    "bound_rank_one_kept": ("rank_one_bound", _b1_kept),
    "bound_factorized_whole_b": ("factorized_bound", _b2_whole_b),
    "bound_normalized_no_sqrt": ("normalized_bound", _bn_no_sqrt),
    "rmsnorm_sum_not_mean": ("rmsnorm", _rms_sum),
    "rmsnorm_eps_outside_sqrt": ("rmsnorm", _rms_eps_outside),
    "rmsnorm_gamma_on_rows": ("rmsnorm", _rms_gamma_rows),
    "rmsnorm_l1": ("rmsnorm", _rms_l1),
    "weights_over_queries": ("attention_weights", _aw_over_queries),
    "weights_unnormalised": ("attention_weights", _aw_unnormalised),
    "weights_masked_row_nan": ("attention_weights", _aw_no_max),
    "rowstats_min": ("softmax_row_stats", _rs_min),
    "rowstats_sum_not_recip": ("softmax_row_stats", _rs_sum_not_recip),
    "rowstats_over_first_axis": ("softmax_row_stats", _rs_over_first_axis),
    "silu_is_sigmoid": ("silu", _silu_sigmoid),
    "silu_sign": ("silu", _silu_sign),
    "swiglu_swapped": ("swiglu", _swiglu_swapped),
    "pv_scores_over_rows": ("reduced_pv", _pv_scores_rows),
    "pv_scores_l1": ("reduced_pv", _pv_scores_l1),
    "pv_gqa_modulo": ("reduced_pv", _pv_gqa_modulo),
    "attn_softmax_over_queries": ("reduced_attention", _attn_over_queries),
    "attn_unnormalised": ("reduced_attention", _attn_unnormalised),
    "attn_mask_as_zero_score": ("reduced_attention", _attn_mask_as_zero),
    "attn_gqa_modulo": ("reduced_attention", _attn_gqa_modulo),
    "k_plain_ceil": ("retained_count", _k_plain_ceil),
    "k_round": ("retained_count", _k_round),
    "k_no_domain_check": ("retained_count", _k_no_domain),
    "energy_l1": ("column_energies", _e_l1),
    "energy_drop_row": ("column_energies", _e_drop_row),
    "energy_rows": ("column_energies", _e_rows),
    "topk_smallest": ("topk_indices", _topk_smallest),
    "topk_ties_high": ("topk_indices", _topk_ties_high),
    "topk_unsorted": ("topk_indices", _topk_unsorted),
    "topk_nan_low": ("topk_indices", _topk_nan_low),
    "matmul_transposed": ("reduced_matmul", _mm_transposed),
    "matmul_off_by_one": ("reduced_matmul", _mm_off_by_one),
    "matmul_sign": ("reduced_matmul", _mm_sign),
    "qk_scale_k": ("reduced_qk", _qk_scale_k),
    "qk_gqa_modulo": ("reduced_qk", _qk_gqa_mod),
    "qk_no_scale": ("reduced_qk", _qk_no_scale),
    "qk_mask_off_by_one": ("reduced_qk", _qk_mask_off_by_one),
    "qk_mask_top_left": ("reduced_qk", _qk_mask_top_left),
    "qk_scores_on_k": ("rmm_qk", _rmm_qk_scores_k),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(ro, attr, fn)
    failed = []
    for check in pins.ALL_CHECKS:
        try:
            check(ro)
        except (AssertionError, ValueError, IndexError, TypeError):
            failed.append(check.__name__)
    assert failed, f"no pin caught mutant {name}"
