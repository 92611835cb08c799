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


def check_index_sets(idx_gpu: np.ndarray, idx_ref: np.ndarray, margins, M: int,
                     exact_sums: bool = False):
    """Bit-exact index sets wherever float64 rounding cannot change the set.

    When the oracle's relative gap at the k boundary is below what two
    float64 summation orders can differ by (and the sums are not exact),
    several sets are correct; then the GPU set must still be a TopK of the
    oracle energies within that rounding bound.  Returns the number of such
    near-tie units (0 in every workload checked so far)."""
    idx_gpu = np.asarray(idx_gpu).reshape(idx_ref.shape)
    near = 0
    for u in range(idx_ref.shape[0]):
        if exact_sums or margins[u] > energy_rel_bound(M):
            assert np.array_equal(idx_gpu[u], idx_ref[u]), (
                f"unit {u}: index set differs (margin {margins[u]:.3e})")
        else:
            near += 1
            assert np.all(np.diff(idx_gpu[u]) > 0)
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


def margins_of(e_ref: np.ndarray, k: int, margin_fn) -> list:
    return [margin_fn(e_ref[u], k) for u in range(e_ref.shape[0])]


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
