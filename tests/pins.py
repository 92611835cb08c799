"""Pins for the CPU oracle: what the paper and mathematics fix, independent of it.

Each ``check_*`` takes the oracle module (or a copy with a planted mistake)
and raises AssertionError when the oracle disagrees with:

* closed forms and exact rational arithmetic (``fractions.Fraction``),
* brute force over all index subsets of tiny inputs (the minimax theorem of
  Appendix E: TopK minimises the residual activation energy),
* special cases that reduce to something known (identity weights, unit-
  vector keys, constant heads),
* the error identity and the bounds of Sec. 3.5 / Appendix E,
* hand-worked fixtures under ``tests/golden``.

These checks never call the HIP library.
"""
from __future__ import annotations

from fractions import Fraction
from itertools import combinations
import math
import os

import numpy as np

import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden_lines(name):
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                yield line.split()


def exact_dot(a, b) -> float:
    """Correctly rounded dot product of two float64 vectors of bf16/fp32 values.

    Each product of two such values is exact in float64 (<= 48 significant
    bits), so fsum of the products is the exact dot product, rounded once.
    """
    return math.fsum(float(x) * float(y) for x, y in zip(a, b))


def exact_matmul(A, B) -> np.ndarray:
    A = np.asarray(A, dtype=np.float64)
    B = np.asarray(B, dtype=np.float64)
    out = np.empty((A.shape[0], B.shape[1]))
    for i in range(A.shape[0]):
        for n in range(B.shape[1]):
            out[i, n] = exact_dot(A[i, :], B[:, n])
    return out


def _bf16(seed, shape, **kw):
    return wl.decode(wl.random_case(seed, shape, "bf16", **kw), "bf16").astype(np.float64)


def _ints(seed, shape, lo, hi):
    return wl.decode(wl.integer_case(seed, shape, lo, hi, "f32"), "f32").astype(np.float64)


# ---------------------------------------------------------------------------
# k = ceil(rho * d)  (Sec. 3.2)
# ---------------------------------------------------------------------------

def check_retained_count(o):
    for r_s, K_s, k_s in _golden_lines("retained_count.txt"):
        got = o.retained_count(float(r_s), int(K_s))
        assert got == int(k_s), (r_s, K_s, got, k_s)
    # ceil of the exact decimal the caller wrote, by rational arithmetic
    for K in (1, 3, 7, 100, 128, 512, 2048, 4096, 8192, 14336, 28672):
        for p in range(1, 101):
            s = f"{p / 100:.2f}"
            want = max(1, math.ceil(Fraction(s) * K))
            got = o.retained_count(float(s), K)
            assert got == want, (s, K, got, want)
    for bad in (0.0, -0.25, 1.0 + 1e-12, 2.0, float("nan"), float("inf"), -float("inf")):
        try:
            o.retained_count(bad, 128)
        except ValueError:
            continue
        raise AssertionError(f"retained_count accepted r={bad}")


# ---------------------------------------------------------------------------
# e_j = ||A[:, j]||^2  (Sec. 3.2)
# ---------------------------------------------------------------------------

def check_energies(o):
    rows = list(_golden_lines("energies_small.txt"))
    A = np.array([[float(v) for v in r[1:]] for r in rows if r[0] == "A"])
    e_want = np.array([float(v) for v in next(r for r in rows if r[0] == "e")[1:]])
    e = o.column_energies(A)
    assert e.dtype == np.float64 and e.shape == (A.shape[1],)
    assert np.array_equal(e, e_want), (e, e_want)
    # exact rational sum of squares, rounded once, for bf16 and fp32 data
    for seed, shape, dt in ((1, (37, 11), "bf16"), (2, (5, 3), "f32"), (3, (64, 7), "bf16")):
        X = wl.decode(wl.random_case(seed, shape, dt, n_outlier=2), dt).astype(np.float64)
        want = np.array([float(sum(Fraction(float(x)) ** 2 for x in X[:, j]))
                         for j in range(shape[1])])
        got = o.column_energies(X)
        assert np.array_equal(got, want), (seed, got - want)
        # Frobenius identity: sum_j e_j = ||A||_F^2
        fro = float(np.linalg.norm(X)) ** 2
        assert abs(math.fsum(got) - fro) <= 1e-12 * fro


# ---------------------------------------------------------------------------
# TopK (Sec. 3.2) vs brute force over subsets (minimax theorem, App. E)
# ---------------------------------------------------------------------------

def brute_force_topk(e_exact, k):
    """Among all size-k subsets, the one with minimum residual energy;
    among those, the lexicographically smallest (ties -> lower indices)."""
    d = len(e_exact)
    best, best_res = None, None
    for S in combinations(range(d), k):          # lexicographic order
        s = set(S)
        res = sum(e_exact[j] for j in range(d) if j not in s)
        if best is None or res < best_res:
            best, best_res = S, res
    return list(best)


def check_selection(o):
    cases = []
    for seed in range(6):
        cases.append(_ints(10 + seed, (4, 9), -3, 3))       # many exact ties
    for seed in range(3):
        cases.append(_ints(20 + seed, (6, 10), -1, 1))      # heavy ties
    cases.append(np.zeros((3, 6)))                          # all-tied zeros
    for A in cases:
        d = A.shape[1]
        # integer data: exact energies without the oracle
        e_exact = [sum(Fraction(int(v)) ** 2 for v in A[:, j]) for j in range(d)]
        e = o.column_energies(A)
        assert [Fraction(float(v)) for v in e] == e_exact
        for k in range(1, d + 1):
            idx = o.topk_indices(e, k)
            got = [int(v) for v in idx]
            assert got == sorted(set(got)) and len(got) == k, got
            assert got == brute_force_topk(e_exact, k), (A, k, got)
    # real-valued bf16 data, nestedness and monotone residual (Sec. 3.5)
    for seed in range(4):
        X = _bf16(30 + seed, (16, 12), n_outlier=2)
        e = o.column_energies(X)
        e_exact = [sum(Fraction(float(x)) ** 2 for x in X[:, j]) for j in range(12)]
        prev_set, prev_res = set(), None
        for k in range(1, 13):
            got = [int(v) for v in o.topk_indices(e, k)]
            assert got == brute_force_topk(e_exact, k)
            assert prev_set <= set(got)
            res = sum(e_exact[j] for j in range(12) if j not in set(got))
            assert prev_res is None or res <= prev_res
            prev_set, prev_res = set(got), res
    # non-finite energies (reading: NaN > inf > finite; NaNs tie)
    rows = list(_golden_lines("nan_ranking.txt"))
    e = np.array([float(v) for v in next(r for r in rows if r[0] == "e")[1:]])
    for r in rows:
        if r[0] == "I":
            k, want = int(r[1]), [int(v) for v in r[2:]]
            assert [int(v) for v in o.topk_indices(e, k)] == want, (k, want)
    # the hand-worked fixture through rmm()
    rowsA = list(_golden_lines("energies_small.txt"))
    A = np.array([[float(v) for v in r[1:]] for r in rowsA if r[0] == "A"])
    for r in rowsA:
        if r[0] == "I":
            _, idx, _ = o.rmm(A, np.eye(4), float(r[1]))
            assert [int(v) for v in idx] == [int(v) for v in r[2:]], r


# ---------------------------------------------------------------------------
# Reduced product (Sec. 3.2 definition; Sec. 3.5 rank-one decomposition)
# ---------------------------------------------------------------------------

def check_product(o):
    # identity weights: RMM(A, I_d) = A with the discarded columns zeroed
    A = _bf16(40, (13, 9))
    idx = np.array([0, 2, 3, 7])
    Y = o.reduced_matmul(A, np.eye(9), idx)
    Z = np.zeros_like(A)
    Z[:, idx] = A[:, idx]
    assert Y.shape == (13, 9) and np.array_equal(Y, Z)
    # cyclic-shift weights (square, not symmetric): row j of B is e_{(j+1) mod d},
    # so column (j+1) mod d of the output is A[:, j] for j in I, else zero
    P = np.zeros((9, 9))
    for j in range(9):
        P[j, (j + 1) % 9] = 1.0
    Y = o.reduced_matmul(A, P, idx)
    Z = np.zeros_like(A)
    for j in idx:
        Z[:, (j + 1) % 9] = A[:, j]
    assert np.array_equal(Y, Z)
    # non-square operands: shape and values against exact dots of the
    # explicitly listed retained rank-one terms
    A = _bf16(41, (7, 11), n_outlier=2)
    B = _bf16(42, (11, 5))
    for idx in (np.array([1, 4, 5, 10]), np.arange(11), np.array([6])):
        Y = o.reduced_matmul(A, B, idx)
        assert Y.shape == (7, 5)
        for i in range(7):
            for n in range(5):
                want = math.fsum(A[i, j] * B[j, n] for j in idx)
                assert abs(Y[i, n] - want) <= 1e-14 * (1 + np.abs(A[i, :]) @ np.abs(B[:, n]))
    # r = 1 is the full product (ceil(1 * d) = d)
    full = exact_matmul(A, B)
    Y1, idx1, _ = o.rmm(A, B, 1.0)
    assert [int(v) for v in idx1] == list(range(11))
    assert np.allclose(Y1, full, rtol=0, atol=1e-13 * np.abs(full).max())
    # complement identity: RMM(I) + RMM(Ibar) = AB (Sec. 3.5)
    for r in (0.25, 0.5, 0.75):
        Yr, idx, _ = o.rmm(A, B, r)
        comp = np.array(sorted(set(range(11)) - set(int(v) for v in idx)))
        Yc = o.reduced_matmul(A, B, comp)
        assert np.allclose(Yr + Yc, full, rtol=0, atol=1e-13 * np.abs(full).max())
    # rmm(): index set is TopK of the column energies, output the product
    X = _bf16(43, (20, 16), n_outlier=3)
    W = _bf16(44, (16, 6))
    Y, idx, e = o.rmm(X, W, 0.5)
    e_exact = [float(sum(Fraction(float(x)) ** 2 for x in X[:, j])) for j in range(16)]
    assert np.array_equal(e, np.array(e_exact))
    assert [int(v) for v in idx] == brute_force_topk([Fraction(v) for v in e_exact], 8)
    # batched: each sequence selects on its own rows (Appendix A)
    Xb = np.stack([_bf16(45, (6, 10), n_outlier=2), _bf16(46, (6, 10), n_outlier=3)])
    Wb = _bf16(47, (10, 4))
    Yb, idxb, eb = o.rmm_batched(Xb, Wb, 0.5)
    for b in range(2):
        Ys, ids, es = o.rmm(Xb[b], Wb, 0.5)
        assert np.array_equal(Yb[b], Ys) and np.array_equal(idxb[b], ids)


def check_bounds(o):
    """Error identity and bounds of Sec. 3.5 / Appendix E hold for the
    oracle's product; the oracle's bound helpers agree with their definition."""
    for seed in range(3):
        A = _bf16(50 + seed, (24, 32), n_outlier=4)
        B = _bf16(60 + seed, (32, 10), std=0.02)
        full = exact_matmul(A, B)
        nA, nB = float(np.linalg.norm(A)), float(np.linalg.norm(B))
        for r in (0.25, 0.5, 0.75, 1.0):
            Y, idx, e = o.rmm(A, B, r)
            comp = sorted(set(range(32)) - set(int(v) for v in idx))
            err = float(np.linalg.norm(full - Y))
            b1 = math.fsum(float(np.linalg.norm(A[:, j]) * np.linalg.norm(B[j, :])) for j in comp)
            b2 = float(np.linalg.norm(A[:, comp]) * np.linalg.norm(B[comp, :])) if comp else 0.0
            epsA = float(np.linalg.norm(A[:, comp]) ** 2) / nA ** 2 if comp else 0.0
            epsB = float(np.linalg.norm(B[comp, :]) ** 2) / nB ** 2 if comp else 0.0
            slack = 1e-12 * nA * nB
            assert err <= b1 + slack
            assert b1 <= b2 * (1 + 1e-12) + slack
            assert err / (nA * nB) <= math.sqrt(epsA * epsB) + 1e-12
            assert abs(o.rank_one_bound(A, B, idx) - b1) <= 1e-12 * (1 + b1)
            assert abs(o.factorized_bound(A, B, idx) - b2) <= 1e-12 * (1 + b2)
            assert abs(o.normalized_bound(A, B, idx) - math.sqrt(epsA * epsB)) <= 1e-12
            assert abs(o.residual_energy(e, idx) - epsA * nA ** 2) <= 1e-10 * nA ** 2
            assert abs(o.retained_energy_fraction(e, idx) - (1 - epsA)) <= 1e-12
            # minimax optimality: any other subset of the same size keeps less energy
            rng = np.random.default_rng(seed)
            for _ in range(20):
                other = rng.choice(32, size=len(idx), replace=False)
                assert o.residual_energy(e, idx) <= o.residual_energy(e, other) + 1e-12


def check_worked_example(o):
    """Appendix E: top 70% of dims hold 95% of the energy -> eps_A(0.7) = 0.05."""
    (rho_s, frac_s, eps_s), = list(_golden_lines("worked_example_appE.txt"))
    rho, frac, eps = float(rho_s), float(frac_s), float(eps_s)
    d, n = 20, 8
    k = 14
    assert math.ceil(Fraction(rho_s) * d) == k
    # 14 strong columns share `frac` of the energy, 6 weak ones the rest
    rng = np.random.default_rng(7)
    A = np.zeros((n, d))
    strong = rng.choice(d, size=k, replace=False)
    weak = [j for j in range(d) if j not in set(strong)]
    for j in strong:
        v = rng.standard_normal(n)
        A[:, j] = v / np.linalg.norm(v) * math.sqrt(frac / k)
    for j in weak:
        v = rng.standard_normal(n)
        A[:, j] = v / np.linalg.norm(v) * math.sqrt((1 - frac) / (d - k))
    B = rng.standard_normal((d, 9))
    Y, idx, e = o.rmm(A, B, rho)
    assert sorted(int(v) for v in idx) == sorted(int(v) for v in strong)
    assert abs(o.discarded_energy_ratio(A, idx, 1) - eps) <= 1e-12
    assert abs(o.retained_energy_fraction(e, idx) - frac) <= 1e-12
    full = A @ B
    epsB = o.discarded_energy_ratio(B, idx, 0)
    rel = np.linalg.norm(full - Y) / (np.linalg.norm(A) * np.linalg.norm(B))
    assert rel <= math.sqrt(eps * epsB) + 1e-12


# ---------------------------------------------------------------------------
# Reduced QK^T (Sec. 3.3)
# ---------------------------------------------------------------------------

def check_qk(o):
    # GQA map: consecutive query heads share a kv head
    assert [o.gqa_kv_head(h, 8, 2) for h in range(8)] == [0, 0, 0, 0, 1, 1, 1, 1]
    assert [o.gqa_kv_head(h, 4, 4) for h in range(4)] == [0, 1, 2, 3]
    # constant heads: S[h,i,t] = k * (g(h) + 1) / sqrt(D)
    H, Hkv, L, D, k = 4, 2, 3, 8, 5
    Q = np.ones((H, L, D))
    K = np.stack([np.full((L, D), g + 1.0) for g in range(Hkv)])
    idx = np.stack([np.arange(k)] * H)
    S = o.reduced_qk(Q, K, idx, causal=False)
    for h in range(H):
        assert np.allclose(S[h], k * (h // 2 + 1) / math.sqrt(D), rtol=1e-15, atol=0)
    # unit-vector keys: S[h,i,t] = Q[h,i,t]/sqrt(D) if t in I_h else 0
    H, L, D = 2, 4, 8
    Q = _bf16(70, (H, L, D))
    K = np.stack([np.eye(D)] * 1)                      # Hkv = 1, Lk = D
    idx = np.array([[0, 3, 5], [1, 2, 7]])
    S = o.reduced_qk(Q, K, idx, causal=False)
    for h in range(H):
        want = np.zeros((L, D))
        want[:, idx[h]] = Q[h][:, idx[h]] / math.sqrt(D)
        assert np.allclose(S[h], want, rtol=1e-15, atol=0)
    # causal mask, Lq=3, Lk=5, bottom-right aligned (hand table)
    mask = np.array([[int(v) for v in r] for r in _golden_lines("causal_mask_3x5.txt")],
                    dtype=bool)
    Q = _bf16(71, (2, 3, 16))
    Kt = _bf16(72, (1, 5, 16))
    idx = np.stack([np.arange(0, 16, 2)] * 2)
    S = o.reduced_qk(Q, Kt, idx, causal=True)
    for h in range(2):
        assert np.array_equal(np.isneginf(S[h]), mask)
        assert np.all(np.isfinite(S[h][~mask]))
    # rows computed one by one are the same rows of the full S, mask included
    Sr = o.reduced_qk(Q, Kt, idx, causal=True, rows=[2, 0])
    assert np.array_equal(Sr[:, 0], S[:, 2]) and np.array_equal(Sr[:, 1], S[:, 0])
    # r = 1 is the dense scaled product (exact dots)
    Q = _bf16(73, (2, 5, 16))
    Kt = _bf16(74, (1, 6, 16))
    S, idx, e = o.rmm_qk(Q, Kt, 1.0, causal=False)
    for h in range(2):
        want = exact_matmul(Q[h], Kt[0].T) / math.sqrt(16)
        assert np.allclose(S[h], want, rtol=0, atol=1e-14 * (1 + np.abs(want).max()))
    # selection is per query head on Q (not on K): integer data, exact energies
    Q = _ints(75, (3, 6, 8), -3, 3)
    Kt = _bf16(76, (1, 7, 8))
    S, idx, e = o.rmm_qk(Q, Kt, 0.5, causal=True)
    for h in range(3):
        e_exact = [sum(Fraction(int(v)) ** 2 for v in Q[h][:, j]) for j in range(8)]
        assert [int(v) for v in idx[h]] == brute_force_topk(e_exact, 4)
        # each head's scores use only its own index set
        want = exact_matmul(Q[h][:, idx[h]], Kt[0][:, idx[h]].T) / math.sqrt(8)
        m = np.triu(np.ones((6, 7), dtype=bool), 2)      # t > i + 1
        assert np.array_equal(np.isneginf(S[h]), m)
        assert np.allclose(S[h][~m], want[~m], rtol=0, atol=1e-14 * (1 + np.abs(want).max()))


def check_attention(o):
    """Reduced attention block (Sec. 3.3): softmax of the reduced, masked
    scores, then the weighted average of the value rows."""
    # two keys, one retained dim: weights 1/(1+e^(s1-s0)) with s_t = a*K[t,0]/sqrt(D);
    # the other dims (5s) would change the result if they were not dropped
    D, a = 4, 1.5
    Q = np.zeros((1, 1, D)); Q[0, 0, 0] = a
    K = np.array([[[1.0, 5, 5, 5], [2.0, 5, 5, 5]]])
    V = np.array([[[1.0, -2.0], [3.0, 4.0]]])
    O = o.reduced_attention(Q, K, V, np.array([[0]]), causal=False)
    s0, s1 = a * 1.0 / math.sqrt(D), a * 2.0 / math.sqrt(D)
    w0 = 1.0 / (1.0 + math.exp(s1 - s0))
    assert np.allclose(O[0, 0], w0 * V[0, 0] + (1 - w0) * V[0, 1], rtol=1e-14, atol=0)
    # all scores equal (Q = 0): the mean of the unmasked value rows (causal
    # prefix means, bottom-right aligned); Lq > Lk leaves fully masked rows at 0
    H, Hkv, Lq, Lk, D = 2, 1, 6, 4, 8
    V = _bf16(80, (Hkv, Lk, 3))
    O = o.reduced_attention(np.zeros((H, Lq, D)), _bf16(81, (Hkv, Lk, D)), V,
                            np.stack([np.arange(4)] * H), causal=True)
    for h in range(H):
        for i in range(Lq):
            n = i + (Lk - Lq) + 1
            want = V[0][:n].mean(axis=0) if n > 0 else np.zeros(3)
            assert np.allclose(O[h, i], want, rtol=1e-14, atol=1e-15)
    # value rows of ones: every row with a key sums its weights to 1
    Q, K = _bf16(82, (3, 5, 16)), _bf16(83, (1, 7, 16))
    idx = np.stack([np.arange(0, 16, 3)] * 3)
    O = o.reduced_attention(Q, K, np.ones((1, 7, 4)), idx, causal=True)
    assert np.allclose(O, 1.0, rtol=1e-14, atol=0)
    # causality: value and key rows past i + (Lk - Lq) do not reach row i
    V = _bf16(84, (1, 7, 4))
    O1 = o.reduced_attention(Q, K, V, idx, causal=True)
    K2, V2 = K.copy(), V.copy()
    K2[0, 6] += 7.0; V2[0, 6] -= 9.0                     # key 6: only row 4 sees it
    O2 = o.reduced_attention(Q, K2, V2, idx, causal=True)
    assert np.array_equal(O1[:, :4], O2[:, :4]) and not np.allclose(O1[:, 4], O2[:, 4])
    # each output lies in the hull of the value rows it averages
    assert np.all(O1 >= V[0].min(axis=0) - 1e-12) and np.all(O1 <= V[0].max(axis=0) + 1e-12)
    # non-causal: permuting key and value rows together changes nothing
    perm = np.array([3, 0, 6, 1, 5, 2, 4])
    Oa = o.reduced_attention(Q, K, V, idx, causal=False)
    Ob = o.reduced_attention(Q, K[:, perm], V[:, perm], idx, causal=False)
    assert np.allclose(Oa, Ob, rtol=1e-13, atol=1e-15)
    # GQA: a query head reads the value rows of kv head h // (H / Hkv)
    V = np.stack([np.full((7, 2), g + 1.0) for g in range(2)])
    O = o.reduced_attention(_bf16(85, (4, 5, 16)), _bf16(86, (2, 7, 16)), V,
                            np.stack([np.arange(6)] * 4), causal=True)
    for h in range(4):
        assert np.allclose(O[h], h // 2 + 1.0, rtol=1e-14, atol=0)
    # rows computed one by one are the same rows
    Or = o.reduced_attention(Q, K, V[:1], idx, causal=True, rows=[4, 1])
    Of = o.reduced_attention(Q, K, V[:1], idx, causal=True)
    assert np.array_equal(Or[:, 0], Of[:, 4]) and np.array_equal(Or[:, 1], Of[:, 1])


def check_pv(o):
    """Token-axis reduced value product (Sec. 3.3): token scores are the
    column norms of each head's weights, the kt strongest tokens are kept."""
    # hand-worked: column energies 0.29, 0.34, 0.25 -> tokens {0, 1}
    P = np.array([[[0.5, 0.5, 0.0], [0.2, 0.3, 0.5]]])
    V = np.array([[[1.0, 2.0], [-1.0, 4.0], [8.0, 8.0]]])
    O, idx = o.reduced_pv(P, V, 2)
    assert idx.tolist() == [[0, 1]]
    assert np.allclose(O[0], [[0.0, 3.0], [-0.1, 1.6]], rtol=0, atol=1e-15)
    # all tokens kept: the dense product (exact dot products, independent of the oracle)
    P, V = _bf16(90, (3, 5, 9)), _bf16(91, (1, 9, 4))
    O, idx = o.reduced_pv(P, V, 9)
    for h in range(3):
        assert np.allclose(O[h], exact_matmul(P[h], V[0]), rtol=1e-14, atol=1e-15)
        assert idx[h].tolist() == list(range(9))
    # brute force: the kept tokens carry the most energy (ties -> lower index),
    # and the dropped part is the sum of the discarded rank-one terms
    for seed in range(4):
        P, V = _ints(92 + seed, (2, 4, 7), -3, 4), _bf16(96 + seed, (2, 7, 3))
        kt = 3
        O, idx = o.reduced_pv(P, V, kt)
        for h in range(2):
            e = [sum(Fraction(int(P[h, q, t])) ** 2 for q in range(4)) for t in range(7)]
            assert idx[h].tolist() == brute_force_topk(e, kt)
            dense = exact_matmul(P[h], V[h])
            rest = sum(np.outer(P[h][:, t], V[h][t]) for t in range(7) if t not in set(idx[h]))
            assert np.allclose(dense - O[h], rest, rtol=1e-12, atol=1e-12)
    # GQA: query head h reads the value rows of kv head h // (H / Hkv)
    P = np.abs(_bf16(100, (4, 3, 6))) + 0.5
    V = np.stack([np.full((6, 2), g + 1.0) for g in range(2)])
    O, idx = o.reduced_pv(P, V, 4)
    for h in range(4):
        rows = P[h][:, idx[h]].sum(axis=1)
        assert np.allclose(O[h], (h // 2 + 1.0) * rows[:, None], rtol=1e-14, atol=0)


def check_swiglu(o):
    # silu(0) = 0; silu(x) - silu(-x) = x (sigmoid(x) + sigmoid(-x) = 1);
    # silu(1) = 1 / (1 + 1/e), silu(-1) = -1 / (1 + e) (closed forms)
    assert o.silu(np.array([0.0]))[0] == 0.0
    xs = np.linspace(-9.0, 9.0, 37)
    assert np.allclose(o.silu(xs) - o.silu(-xs), xs, rtol=0, atol=1e-14)
    assert abs(o.silu(np.array([1.0]))[0] - 1.0 / (1.0 + math.exp(-1.0))) < 1e-16
    assert abs(o.silu(np.array([-1.0]))[0] + 1.0 / (1.0 + math.e)) < 1e-16
    # tails: x for large x, 0 from below for very negative x
    assert o.silu(np.array([40.0]))[0] == 40.0
    v = o.silu(np.array([-40.0]))[0]
    assert -1e-15 < v < 0.0
    # the activation gates with g and scales by u (not the other way round)
    g, u = np.array([1.0, -2.0, 3.0]), np.array([2.0, 0.5, -1.0])
    want = np.array([2.0 / (1.0 + math.exp(-1.0)), 0.5 * -2.0 / (1.0 + math.exp(2.0)),
                     -3.0 / (1.0 + math.exp(-3.0))])
    assert np.allclose(o.swiglu(g, u), want, rtol=1e-15, atol=0)


def check_rmsnorm(o):
    # hand-worked: x = (3, 4), gamma = (1, 2), eps = 0: mean of squares 12.5,
    # y = (3, 8) / sqrt(12.5)
    y = o.rmsnorm(np.array([[3.0, 4.0]]), np.array([1.0, 2.0]), 0.0)
    assert np.allclose(y, np.array([[3.0, 8.0]]) / math.sqrt(12.5), rtol=1e-15, atol=0)
    # with gamma = 1 and eps = 0 every row has mean square exactly 1 (closed
    # form), whatever its scale; rows are independent of each other
    rng = np.random.default_rng(5)
    X = rng.standard_normal((6, 10)) * np.array([1e-3, 1, 7, 50, 0.2, 3])[:, None]
    Y = o.rmsnorm(X, np.ones(10), 0.0)
    assert np.allclose((Y * Y).mean(axis=1), 1.0, rtol=1e-14, atol=0)
    assert np.allclose(o.rmsnorm(X * 5.0, np.ones(10), 0.0), Y, rtol=1e-14, atol=0)
    assert np.allclose(o.rmsnorm(X[3:4], np.ones(10), 0.0), Y[3:4], rtol=1e-15, atol=0)
    # gamma scales columns (channels), not rows
    g = np.arange(1.0, 11.0)
    assert np.allclose(o.rmsnorm(X, g, 0.0), Y * g[None, :], rtol=1e-14, atol=0)
    # eps sits inside the square root: a constant row c gives c / sqrt(c^2 + eps)
    y = o.rmsnorm(np.full((1, 4), 2.0), np.ones(4), 5.0)
    assert np.allclose(y, 2.0 / 3.0, rtol=1e-15, atol=0)
    # an all-zero row stays zero (eps > 0)
    assert np.array_equal(o.rmsnorm(np.zeros((1, 3)), np.ones(3), 1e-6), np.zeros((1, 3)))


def check_attention_weights(o):
    # two keys: the weights are the logistic function of the score gap
    P = o.attention_weights(np.array([[0.0, math.log(3.0)]]))
    assert np.allclose(P, [[0.25, 0.75]], rtol=1e-15, atol=0)
    # each row sums to 1 over its kept keys, masked keys get exactly 0, and a
    # row with every key masked is all zeros
    S = np.array([[1.0, -np.inf, 2.0, 0.5], [-np.inf] * 4, [3.0, 3.0, 3.0, -np.inf]])
    P = o.attention_weights(S)
    assert P[0, 1] == 0.0 and P[2, 3] == 0.0 and np.array_equal(P[1], np.zeros(4))
    assert np.allclose(P[[0, 2]].sum(axis=1), 1.0, rtol=1e-15, atol=0)
    assert np.allclose(P[2, :3], 1.0 / 3.0, rtol=1e-15, atol=0)
    e = np.exp([1.0, 2.0, 0.5])
    assert np.allclose(P[0, [0, 2, 3]], e / e.sum(), rtol=1e-15, atol=0)
    # shift invariance per row, and the normalisation runs over keys (last
    # axis), not over queries
    rng = np.random.default_rng(6)
    S = rng.standard_normal((2, 3, 5))
    assert np.allclose(o.attention_weights(S + 7.0), o.attention_weights(S), rtol=1e-13, atol=0)
    assert np.allclose(o.attention_weights(S).sum(axis=-1), 1.0, rtol=1e-14, atol=0)


def check_softmax_row_stats(o):
    # two keys 0 and ln 3: the maximum is ln 3 and the sum 1/3 + 1
    m, rinv = o.softmax_row_stats(np.array([[0.0, math.log(3.0)]]))
    assert m[0] == math.log(3.0) and abs(rinv[0] - 0.75) <= 1e-15
    # n equal scores: 1/n; masked keys do not count; an empty row is (0, 0);
    # the maximum is taken over the kept keys only
    S = np.array([[2.5, 2.5, 2.5, 2.5], [1.0, -np.inf, 1.0, -np.inf], [-np.inf] * 4,
                  [-7.0, -np.inf, -9.0, -np.inf]])
    m, rinv = o.softmax_row_stats(S)
    assert list(m) == [2.5, 1.0, 0.0, -7.0]
    assert np.allclose(rinv, [0.25, 0.5, 0.0, 1.0 / (1.0 + math.exp(-2.0))], rtol=1e-15, atol=0)
    # statistics over the last axis: a [2, 3, 5] input gives [2, 3] pairs; the
    # maximum moves with a shift, the sum does not
    rng = np.random.default_rng(8)
    S = rng.standard_normal((2, 3, 5))
    m, rinv = o.softmax_row_stats(S)
    assert m.shape == (2, 3) and np.array_equal(m, S.max(axis=-1))
    m2, rinv2 = o.softmax_row_stats(S + 4.0)
    assert np.allclose(m2, m + 4.0, rtol=0, atol=1e-14) and np.allclose(rinv2, rinv, rtol=1e-14, atol=0)
    # with a brute-force sum of exp(s - m) over the row
    for i in range(2):
        for j in range(3):
            tot = sum(math.exp(float(v) - float(m[i, j])) for v in S[i, j])
            assert abs(rinv[i, j] * tot - 1.0) <= 1e-14


def check_bound_values(o):
    """The bound helpers on small integer cases whose values are worked out
    by hand (not from the helpers' formulas), Sec. 3.5 / Appendix E.

    Case 1: one discarded column, so the error is the rank-one term
    A[:, 1] B[1, :] and both bounds are tight: ||(0, 4)|| * ||(0, 2)|| = 8.
    eps_A = 16 / 25 (column 1 carries 16 of A's 25), eps_B = 4 / 31.

    Case 2: columns 0 and 1 discarded, a0 = (1, 0), a1 = (0, 2) and rows
    b0 = (1, 0), b1 = (0, 3): error ||a0 b0^T + a1 b1^T|| = ||diag(1, 6)|| =
    sqrt(37); rank-one bound 1*1 + 2*3 = 7; factorized bound
    sqrt(1 + 4) * sqrt(1 + 9) = sqrt(50); eps_A = 5 / 13, eps_B = 10 / 12."""
    A1 = np.array([[3.0, 0.0, 0.0], [0.0, 4.0, 0.0]])
    B1 = np.array([[1.0, 1.0], [0.0, 2.0], [5.0, 0.0]])
    i1 = np.array([0, 2])
    assert o.rank_one_bound(A1, B1, i1) == 8.0
    assert o.factorized_bound(A1, B1, i1) == 8.0
    assert abs(o.normalized_bound(A1, B1, i1) - math.sqrt(16 / 25 * 4 / 31)) <= 1e-15
    Y1, e1 = o.reduced_matmul(A1, B1, i1), o.column_energies(A1)
    assert float(np.linalg.norm(exact_matmul(A1, B1) - Y1)) == 8.0
    assert o.residual_energy(e1, i1) == 16.0
    assert o.retained_energy_fraction(e1, i1) == 9.0 / 25.0

    A2 = np.array([[1.0, 0.0, 2.0], [0.0, 2.0, 2.0]])
    B2 = np.array([[1.0, 0.0], [0.0, 3.0], [1.0, 1.0]])
    i2 = np.array([2])
    assert o.rank_one_bound(A2, B2, i2) == 7.0
    assert abs(o.factorized_bound(A2, B2, i2) - math.sqrt(50.0)) <= 1e-14
    assert abs(o.normalized_bound(A2, B2, i2) - math.sqrt(5 / 13 * 10 / 12)) <= 1e-15
    Y2 = o.reduced_matmul(A2, B2, i2)
    assert abs(float(np.linalg.norm(exact_matmul(A2, B2) - Y2)) - math.sqrt(37.0)) <= 1e-14
    assert o.residual_energy(o.column_energies(A2), i2) == 5.0


def check_margin(o):
    assert o.selection_margin(np.array([4.0, 2.0, 1.0]), 1) == 0.5
    assert o.selection_margin(np.array([4.0, 4.0, 1.0]), 1) == 0.0
    assert o.selection_margin(np.array([4.0, 2.0, 1.0]), 3) == math.inf
    assert o.selection_margin(np.array([1.0, 3.0, 2.0]), 2) == 0.5


ALL_CHECKS = (check_retained_count, check_energies, check_selection, check_product,
              check_bounds, check_worked_example, check_qk, check_attention, check_pv,
              check_swiglu, check_rmsnorm, check_attention_weights, check_softmax_row_stats,
              check_bound_values, check_margin)
