"""Helpers for the GPU parity tests: device copies of stored inputs and the
comparison rules (bit-exact index sets; error bounds derived from the
arithmetic for floating-point outputs)."""
from __future__ import annotations

import numpy as np
import pytest
import torch

U64 = 2.0 ** -53     # float64 unit roundoff
U32 = 2.0 ** -24     # fp32 unit roundoff
U16 = 2.0 ** -8      # bf16 unit roundoff (8-bit significand)

# spec tolerances on the normalised max error max|Y - Y_ref| / max|Y_ref|
NORM_TOL = {"bf16": 2e-2, "f32": 1e-5}

gpu = pytest.mark.gpu


def require_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    return torch.device("cuda:0")


def to_device(stored: np.ndarray, dtype: str, dev) -> torch.Tensor:
    """Device tensor holding exactly the stored bytes (bf16 bits or fp32)."""
    if dtype == "bf16":
        return torch.from_numpy(stored.view(np.int16)).to(dev).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(stored, dtype=np.float32)).to(dev)


def from_device(t: torch.Tensor) -> np.ndarray:
    """float64 values of a bf16/fp32 device tensor."""
    return t.float().cpu().numpy().astype(np.float64)


def torch_dtype(dtype: str):
    return torch.bfloat16 if dtype == "bf16" else torch.float32


def check_energies(e_gpu: np.ndarray, e_ref: np.ndarray, M: int):
    """GPU float64 sums of M exact squares (any order) vs the correctly rounded
    exact sum: |e_gpu - e| <= (M - 1) u e and |e_ref - e| <= u e."""
    e_gpu = np.asarray(e_gpu, dtype=np.float64)
    fin = np.isfinite(e_ref)
    assert np.array_equal(np.isnan(e_gpu), np.isnan(e_ref))
    assert np.array_equal(np.isposinf(e_gpu), np.isposinf(e_ref))
    tol = (M + 1) * U64 * np.abs(e_ref[fin]) * (1 + 1e-9)
    err = np.abs(e_gpu[fin] - e_ref[fin])
    assert np.all(err <= tol), f"energy error {np.max(err - tol)} above bound"


def energy_rel_bound(M: int) -> float:
    return 2 * (M + 1) * U64


def _order_value(e: np.ndarray) -> np.ndarray:
    """Energies as ranking values: NaN above +inf above every finite value."""
    v = np.asarray(e, dtype=np.float64).copy()
    v[np.isnan(v)] = np.inf
    return v


def _boundary_gap(e: np.ndarray, k: int):
    """(a, b): the k-th and (k+1)-th largest ranking values of one unit
    (b = None when k == K).  NaN and +inf rank as +inf."""
    v = np.sort(_order_value(e))[::-1]
    return float(v[k - 1]), (float(v[k]) if k < v.shape[0] else None)


def is_near_tie(e: np.ndarray, k: int, M: int) -> bool:
    """True when two float64 summation orders of M squares could order the
    k-th and (k+1)-th energies differently: their exact gap is at most the
    rounding bound 2(M+1)u of the larger one (an equal pair of rounded sums
    included: their exact sums may still differ).  Ties at +inf or NaN come
    from the inputs themselves and are decided by the index rule alone."""
    a, b = _boundary_gap(e, k)
    if b is None or not np.isfinite(a):
        return False
    return (a - b) <= energy_rel_bound(M) * a


def check_index_sets(idx_gpu, idx_ref: np.ndarray, e_ref, M: int,
                     exact_sums: bool = False, max_near: int = 0):
    """Bit-exact index sets wherever float64 rounding cannot change the set.

    idx_ref [U x k] are the oracle's sets, e_ref [U x K] the oracle's energies
    (exact sums rounded once) of the same units.  Every GPU list must hold k
    strictly ascending indices in [0, K).  Where the oracle's gap at the k
    boundary exceeds what two float64 summation orders of M squares can
    differ by (or the sums are exact), the list must equal the oracle's.
    Otherwise (a near tie) several sets are correct and the list must be a
    TopK of the oracle energies within that bound:
        min(e[kept]) >= max(e[dropped]) - 2(M+1)u * max(min(e[kept]), max(e[dropped])).
    At most ``max_near`` units may be near ties (None: no limit).  Returns
    the number of near-tie units."""
    idx_ref = np.asarray(idx_ref)
    U, k = idx_ref.shape
    e_ref = np.asarray(e_ref, dtype=np.float64).reshape(U, -1)
    K = e_ref.shape[1]
    idx_gpu = np.asarray(idx_gpu).reshape(-1)
    assert idx_gpu.shape[0] == U * k, f"expected {U} lists of {k} indices, got {idx_gpu.shape[0]} values"
    idx_gpu = idx_gpu.reshape(U, k).astype(np.int64)
    near = 0
    for u in range(U):
        g = idx_gpu[u]
        assert np.all((g >= 0) & (g < K)), f"unit {u}: index outside [0, {K})"
        assert np.all(np.diff(g) > 0), f"unit {u}: list not strictly ascending"
        if exact_sums or not is_near_tie(e_ref[u], k, M):
            assert np.array_equal(g, idx_ref[u]), f"unit {u}: index set differs from the oracle"
            continue
        near += 1
        v = _order_value(e_ref[u])
        kept = np.zeros(K, dtype=bool)
        kept[g] = True
        if kept.all():
            continue
        lo, hi = float(v[kept].min()), float(v[~kept].max())
        tol = energy_rel_bound(M) * max(lo, hi)
        assert lo >= hi - tol, (
            f"unit {u}: not a TopK within the float64 bound (kept min {lo:.17g}, "
            f"dropped max {hi:.17g})")
    if max_near is not None:
        assert near <= max_near, f"{near} near-tie units (at most {max_near} allowed)"
    if near:
        print(f"check_index_sets: {near} of {U} units within float64 rounding of a tie", flush=True)
    return near


def bound_matrix(A_abs: np.ndarray, B_abs: np.ndarray) -> np.ndarray:
    return A_abs @ B_abs


def check_product(Y_gpu: np.ndarray, Y_ref: np.ndarray, absprod: np.ndarray, k: int,
                  dtype: str, scale: float = 1.0):
    """Elementwise bound + spec normalised max error.

    fp32 accumulation of k exact products (any order) errs by at most
    k u32 sum|x w|; the fp32 rounding of `scale`, the multiply by it and the
    rounding to the output type add one relative rounding each (u16 for a
    bf16 output, u32 for fp32).
    """
    u_out = U16 if dtype == "bf16" else U32
    acc = (k + 2) * U32 * np.abs(scale) * absprod
    tol = (u_out + 2 * U32) * np.abs(Y_ref) + acc * (1 + u_out) + 1e-300
    err = np.abs(Y_gpu - Y_ref)
    bad = err > tol
    assert not bad.any(), (
        f"{int(bad.sum())} outputs outside the rounding bound; worst excess "
        f"{float(np.max(err - tol)):.3e}")
    norm = float(np.max(err) / max(np.max(np.abs(Y_ref)), 1e-300))
    assert norm <= NORM_TOL[dtype], f"normalised max error {norm:.3e}"
    return norm


def isclose_inf_pattern(S_gpu: np.ndarray, S_ref: np.ndarray):
    assert np.array_equal(np.isneginf(S_gpu), np.isneginf(S_ref))
    assert np.all(np.isfinite(S_gpu[~np.isneginf(S_ref)]))



def attention_bound(Q: np.ndarray, K: np.ndarray, V: np.ndarray, idx: np.ndarray, causal: bool,
                    scale: float, rows=None) -> np.ndarray:
    """Per-row bound on |O - O_ref| for the reduced attention block.

    Each weight carries its bf16 rounding (2^-9 relative) and the fp32 error
    of its score, (k + 4) u32 |scale| sum|q||k| (accumulation, the scale and
    the exponent argument), which moves it by a factor exp(+-2 err); the
    output is then within 2 d max|V| of the reference, d the largest of those
    relative moves.  Q [H x Lq x D], K, V [Hkv x Lk x D], idx [H x k] in
    float64; ``rows`` selects query rows (default all).  Rows with every key
    masked get 0 (their output must be exactly 0).
    """
    H, Lq, _ = Q.shape
    Hkv, Lk, _ = K.shape
    k = idx.shape[1]
    rows = np.arange(Lq) if rows is None else np.asarray(rows)
    out = np.empty((H, rows.shape[0]))
    for h in range(H):
        g = h // (H // Hkv)
        I = idx[h]
        mag = np.abs(Q[h][rows][:, I]) @ np.abs(K[g][:, I]).T          # [rows, Lk]
        err_s = (k + 4) * U32 * abs(scale) * mag
        for n, i in enumerate(rows):
            keep = np.arange(Lk) <= (i + Lk - Lq) if causal else np.ones(Lk, bool)
            if not keep.any():
                out[h, n] = 0.0
                continue
            d = np.expm1(2.0 ** -9 + 2.0 * err_s[n][keep].max())
            out[h, n] = 2.0 * d * np.abs(V[g][keep]).max()
    return out
