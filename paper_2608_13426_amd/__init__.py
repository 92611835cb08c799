"""Python binding of librmm (Reduced Matrix Multiplication on MI355X).

Thin ctypes layer over the C-ABI declared in ``include/rmm.h``: it reads
sizes and strides off torch tensors, passes raw device pointers and the
current HIP stream, and raises ``RmmError`` on a non-zero status.  Every
step of the computation runs in librmm's gfx950 kernels; torch only owns the
device memory and the stream.  Importing this package fails loudly when
``librmm.so`` has not been built (``python paper_2608_13426_amd/build.py``).
"""
from __future__ import annotations

import ctypes
import os

import torch

__all__ = [
    "RmmError", "LIB_PATH", "lib", "RMM_F32", "RMM_BF16", "RMM_OP_SCORE",
    "RMM_OP_SELECT", "RMM_OP_LINEAR", "RMM_OP_ATTENTION", "RMM_OP_PV", "rmm_retained_count",
    "rmm_workspace_size", "rmm_reduced_pv",
    "rmm_status_string", "rmm_score", "rmm_select", "rmm_reduced_gemm",
    "rmm_reduced_qk", "rmm_linear", "rmm_score_kmajor", "rmm_reduced_gemm_kmajor",
    "rmm_reduced_attention", "rmm_reduced_gemv", "rmm_gemv_workspace_size", "rmm_select_tokens",
    "rmm_linear_noalloc", "rmm_noalloc_scratch_bytes", "rmm_rmsnorm_kmajor",
    "rmm_rmsnorm_kmajor_workspace_size", "rmm_attention_weights_kmajor",
    "rmm_attention_weights_kmajor_workspace_size", "rmm_reduced_pv_kmajor", "rmm_decode_step",
    "rmm_decode_step_workspace_size", "rmm_decode_products", "rmm_decode_products_shared",
    "rmm_decode_products_shared_workspace_size", "rmm_decode_step_shared", "DecodeGroup",
    "rmm_reduced_qk_rowstats",
    "rmm_attention_weights_kmajor_rowstats", "EXPORTED_SYMBOLS",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "librmm.so")

RMM_F32, RMM_BF16 = 0, 1
RMM_OP_SCORE, RMM_OP_SELECT, RMM_OP_LINEAR, RMM_OP_ATTENTION, RMM_OP_PV = 0, 1, 2, 3, 4

_p = ctypes.c_void_p
_i64 = ctypes.c_int64


class DecodeGroup(ctypes.Structure):
    """rmm_decode_group_t: one projection group of a decode step."""
    _fields_ = [("X", _p), ("W", _p), ("idx", _p), ("Y", _p), ("K", _i64), ("N", _i64),
                ("k", _i64), ("ldx", _i64), ("ldw", _i64), ("ldy", _i64)]
_SIGS = {
    "rmm_retained_count": (_i64, [ctypes.c_double, _i64]),
    "rmm_workspace_size": (ctypes.c_size_t, [ctypes.c_int, _i64, _i64, _i64, _i64]),
    "rmm_score": (ctypes.c_int, [_p, ctypes.c_int, _i64, _i64, _i64, _i64, _p, _p,
                                 ctypes.c_size_t, _p]),
    "rmm_select": (ctypes.c_int, [_p, _i64, _i64, _i64, _p, _p]),
    "rmm_reduced_gemm": (ctypes.c_int, [_p, _p, _p, ctypes.c_int, _i64, _i64, _i64, _i64,
                                        _i64, _i64, _i64, _p, _i64, _p]),
    "rmm_gemv_workspace_size": (ctypes.c_size_t, [_i64, _i64, _i64, _i64]),
    "rmm_select_tokens": (ctypes.c_int, [_p, ctypes.c_int, _i64, _i64, _i64, _i64, _p, _p]),
    "rmm_reduced_gemv": (ctypes.c_int, [_p, _p, _p, ctypes.c_int, _i64, _i64, _i64, _i64,
                                        _i64, _i64, _i64, _p, _i64, _p, ctypes.c_size_t, _p]),
    "rmm_reduced_qk": (ctypes.c_int, [_p, _p, _p, ctypes.c_int, _i64, _i64, _i64, _i64, _i64,
                                      _i64, _i64, ctypes.c_float, ctypes.c_int, _p, _p]),
    "rmm_linear": (ctypes.c_int, [_p, _p, ctypes.c_double, ctypes.c_int, _i64, _i64, _i64,
                                  _i64, _i64, _i64, _p, _i64, _p, _p, ctypes.c_size_t, _p]),
    "rmm_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "rmm_noalloc_scratch_bytes": (ctypes.c_size_t, []),
    "rmm_rmsnorm_kmajor_workspace_size": (ctypes.c_size_t, [_i64, _i64, _i64]),
    "rmm_attention_weights_kmajor_workspace_size": (ctypes.c_size_t, [_i64, _i64, _i64, _i64]),
    "rmm_attention_weights_kmajor": (ctypes.c_int, [_p, _i64, _i64, _i64, _i64, _i64, ctypes.c_int,
                                                    _p, _i64, _p, _p, ctypes.c_size_t, _p]),
    "rmm_reduced_qk_rowstats": (ctypes.c_int, [_p, _p, _p, _i64, _i64, _i64, _i64, _i64, _i64, _i64,
                                               ctypes.c_float, ctypes.c_int, _p, _p, _p, _p]),
    "rmm_attention_weights_kmajor_rowstats": (ctypes.c_int, [_p, _i64, _i64, _i64, _i64, _i64,
                                                             ctypes.c_int, _p, _p, _p, _i64, _p, _p,
                                                             ctypes.c_size_t, _p]),
    "rmm_decode_step_workspace_size": (ctypes.c_size_t, [ctypes.POINTER(DecodeGroup), ctypes.c_int,
                                                         _i64]),
    "rmm_decode_step": (ctypes.c_int, [ctypes.POINTER(DecodeGroup), ctypes.c_int, _i64, _p,
                                       ctypes.c_size_t, _p]),
    "rmm_decode_products": (ctypes.c_int, [ctypes.POINTER(DecodeGroup), ctypes.c_int, _i64, _p,
                                       ctypes.c_size_t, _p]),
    "rmm_decode_products_shared_workspace_size": (ctypes.c_size_t, [ctypes.POINTER(DecodeGroup),
                                                                    ctypes.c_int, _i64]),
    "rmm_decode_products_shared": (ctypes.c_int, [ctypes.POINTER(DecodeGroup), ctypes.c_int, _i64,
                                                  _p, ctypes.c_size_t, _p]),
    "rmm_decode_step_shared": (ctypes.c_int, [ctypes.POINTER(DecodeGroup), ctypes.c_int, _i64, _p,
                                              ctypes.c_size_t, _p]),
    "rmm_reduced_pv_kmajor": (ctypes.c_int, [_p, _p, _p, _i64, _i64, _i64, _i64, _i64, _i64, _i64,
                                             _i64, ctypes.c_int, _p, _p]),
    "rmm_rmsnorm_kmajor": (ctypes.c_int, [_p, _p, ctypes.c_float, _i64, _i64, _i64, _i64, _p, _i64,
                                          _p, _p, ctypes.c_size_t, _p]),
    "rmm_linear_noalloc": (ctypes.c_int, [_p, _p, ctypes.c_double, ctypes.c_int, _i64, _i64, _i64,
                                          _i64, _i64, _i64, _p, _i64, _p, _p]),
    "rmm_score_kmajor": (ctypes.c_int, [_p, _i64, _i64, _i64, _i64, _p, _p, _i64, _p,
                                        ctypes.c_size_t, _p]),
    "rmm_reduced_gemm_kmajor": (ctypes.c_int, [_p, _p, _p, _i64, _i64, _i64, _i64, _i64, _i64,
                                               _i64, _p, _i64, _p]),
    "rmm_reduced_attention": (ctypes.c_int, [_p, _p, _p, _p, ctypes.c_int, _i64, _i64, _i64, _i64,
                                             _i64, _i64, _i64, ctypes.c_float, ctypes.c_int, _p,
                                             _p, ctypes.c_size_t, _p]),
    "rmm_reduced_pv": (ctypes.c_int, [_p, _p, ctypes.c_int, _i64, _i64, _i64, _i64, _i64, _i64,
                                      _i64, _i64, _p, _p, _p, ctypes.c_size_t, _p]),
    "rmm_attention_kmajor_workspace_size": (ctypes.c_size_t, [_i64, _i64, _i64, _i64, _i64, _i64]),
    "rmm_gemm_swiglu_workspace_size": (ctypes.c_size_t, [_i64, _i64, _i64]),
    "rmm_check_indices": (ctypes.c_int, [_p, _i64, _i64, _i64, _p, _p]),
    "rmm_reduced_gemm_swiglu_kmajor": (ctypes.c_int, [_p, _p, _p, _i64, _i64, _i64, _i64, _i64,
                                                      _i64, _i64, _p, _i64, _p, _p,
                                                      ctypes.c_size_t, _p]),
    "rmm_reduced_attention_kmajor": (ctypes.c_int, [_p, _p, _p, _p, ctypes.c_int, _i64, _i64, _i64,
                                                    _i64, _i64, _i64, _i64, ctypes.c_float,
                                                    ctypes.c_int, _p, _i64, _p, _p, ctypes.c_size_t,
                                                    _p]),
}
EXPORTED_SYMBOLS = tuple(_SIGS)


class RmmError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__(f"{fn} failed: {rmm_status_string(status)} (status {status})")


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"librmm.so is missing at {LIB_PATH}; build it with "
                          "`python paper_2608_13426_amd/build.py`")
    handle = ctypes.CDLL(LIB_PATH)
    for name, (res, args) in _SIGS.items():
        fn = getattr(handle, name)
        fn.restype = res
        fn.argtypes = args
    return handle


lib = _load()


# ---------------------------------------------------------------- helpers

def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return RMM_BF16
    if t.dtype == torch.float32:
        return RMM_F32
    raise TypeError(f"unsupported dtype {t.dtype}; librmm takes bfloat16 or float32")


def _dev(*ts: torch.Tensor) -> torch.device:
    d = ts[0].device
    for t in ts:
        if t.device.type != "cuda":
            raise ValueError("librmm tensors must live on the GPU")
        if t.device != d:
            raise ValueError("all tensors must be on one device")
    return d


def _stream(device: torch.device, stream) -> int:
    s = torch.cuda.current_stream(device) if stream is None else stream
    return s.cuda_stream


def _ptr(t):
    return None if t is None else t.data_ptr()


def _rows(t: torch.Tensor, name: str):
    """View a [U, M, K] or [M, K] tensor as U units of M rows with stride ldx."""
    if t.dim() == 2:
        t3 = t.unsqueeze(0)
    elif t.dim() == 3:
        t3 = t
    else:
        raise ValueError(f"{name} must be 2-D or 3-D")
    U, M, K = t3.shape
    if t3.stride(2) != 1:
        raise ValueError(f"{name} rows must be contiguous")
    ldx = t3.stride(1)
    if U > 1 and t3.stride(0) != M * ldx:
        raise ValueError(f"{name} units must be packed (stride M*ldx)")
    return U, M, K, ldx


def _check(fn: str, status: int):
    if status != 0:
        raise RmmError(fn, status)


# ---------------------------------------------------------------- C-ABI

def rmm_retained_count(r: float, K: int) -> int:
    """k = ceil(r*K) (Sec. 3.2); -1 for r outside (0, 1] or K < 1."""
    return int(lib.rmm_retained_count(float(r), int(K)))


def rmm_workspace_size(op: int, B: int, M: int, K: int, k: int = 0) -> int:
    return int(lib.rmm_workspace_size(int(op), int(B), int(M), int(K), int(k)))


def rmm_status_string(status: int) -> str:
    return lib.rmm_status_string(int(status)).decode()


def rmm_score(X: torch.Tensor, energy: torch.Tensor, workspace: torch.Tensor | None = None,
              stream=None) -> torch.Tensor:
    """Column energies of each unit of X ([B, M, K] or [M, K]) into float64 energy [B, K]."""
    B, M, K, ldx = _rows(X, "X")
    d = _dev(X, energy)
    if energy.dtype != torch.float64 or energy.numel() != B * K or not energy.is_contiguous():
        raise ValueError("energy must be a contiguous float64 tensor of B*K elements")
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check("rmm_score", lib.rmm_score(X.data_ptr(), _dtype_code(X), B, M, K, ldx,
                                      energy.data_ptr(), _ptr(workspace), ws_bytes,
                                      _stream(d, stream)))
    return energy


def rmm_score_kmajor(X: torch.Tensor, energy: torch.Tensor, Xt: torch.Tensor,
                     workspace: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Energies of each unit of bf16 X [B, M, K] plus its K-major copy Xt [B, K, ldxt]."""
    B, M, K, ldx = _rows(X, "X")
    d = _dev(X, energy, Xt)
    if energy.dtype != torch.float64 or energy.numel() != B * K or not energy.is_contiguous():
        raise ValueError("energy must be a contiguous float64 tensor of B*K elements")
    Bt, Kt, Mt, ldxt = _rows(Xt, "Xt")
    if (Bt, Kt, Mt) != (B, K, M) or Xt.dtype != X.dtype:
        raise ValueError("Xt must be [B, K, M] (a view with row stride ldxt) of X's dtype")
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check("rmm_score_kmajor", lib.rmm_score_kmajor(
        X.data_ptr(), B, M, K, ldx, energy.data_ptr(), Xt.data_ptr(), ldxt, _ptr(workspace),
        ws_bytes, _stream(d, stream)))
    return energy


def rmm_select(energy: torch.Tensor, k: int, idx: torch.Tensor, stream=None) -> torch.Tensor:
    """TopK (ascending int32 indices) of each unit's energies.

    energy holds B units of K float64 energies ([B, K], or flat); idx holds
    B*k int32 slots, from which B is read.
    """
    d = _dev(energy, idx)
    k = int(k)
    if energy.dtype != torch.float64 or not energy.is_contiguous():
        raise ValueError("energy must be contiguous float64")
    if idx.dtype != torch.int32 or not idx.is_contiguous() or k < 1 or idx.numel() % k:
        raise ValueError("idx must be a contiguous int32 tensor of B*k elements")
    B = idx.numel() // k
    if B < 1 or energy.numel() % B:
        raise ValueError("energy must hold B*K values")
    K = energy.numel() // B
    _check("rmm_select", lib.rmm_select(energy.data_ptr(), B, K, k, idx.data_ptr(),
                                        _stream(d, stream)))
    return idx


def rmm_reduced_gemm(X: torch.Tensor, W: torch.Tensor, idx: torch.Tensor, Y: torch.Tensor,
                     stream=None) -> torch.Tensor:
    """Y[b] = X[b][:, I_b] @ W[I_b, :] for X [B, M, K], W [K, N], idx [B, k], Y [B, M, N]."""
    B, M, K, ldx = _rows(X, "X")
    d = _dev(X, W, idx, Y)
    if W.dim() != 2 or W.shape[0] != K or W.stride(1) != 1:
        raise ValueError("W must be [K, N] with contiguous rows")
    N, ldw = W.shape[1], W.stride(0)
    By, My, Ny, ldy = _rows(Y, "Y")
    if (By, My, Ny) != (B, M, N):
        raise ValueError("Y must be [B, M, N]")
    if not (X.dtype == W.dtype == Y.dtype):
        raise TypeError("X, W and Y must share one dtype")
    if idx.dtype != torch.int32 or not idx.is_contiguous() or idx.numel() % B:
        raise ValueError("idx must be contiguous int32 [B, k]")
    k = idx.numel() // B
    _check("rmm_reduced_gemm", lib.rmm_reduced_gemm(
        X.data_ptr(), W.data_ptr(), idx.data_ptr(), _dtype_code(X), B, M, N, K, k, ldx, ldw,
        Y.data_ptr(), ldy, _stream(d, stream)))
    return Y


def rmm_check_indices(idx: torch.Tensor, K: int, bad: torch.Tensor | None = None,
                      stream=None) -> torch.Tensor:
    """Per unit of idx [B, k]: 0 if its list is strictly ascending within
    [0, K), else 1 + the first position that breaks it (int32 [B])."""
    if idx.dim() == 1:
        idx = idx.unsqueeze(0)
    if idx.dtype != torch.int32 or not idx.is_contiguous() or idx.dim() != 2:
        raise ValueError("idx must be contiguous int32 [B, k]")
    B, k = idx.shape
    if bad is None:
        bad = torch.empty(B, dtype=torch.int32, device=idx.device)
    d = _dev(idx, bad)
    if bad.dtype != torch.int32 or bad.numel() != B or not bad.is_contiguous():
        raise ValueError("bad must be contiguous int32 [B]")
    _check("rmm_check_indices", lib.rmm_check_indices(idx.data_ptr(), B, k, int(K), bad.data_ptr(),
                                                      _stream(d, stream)))
    return bad


def rmm_select_tokens(X: torch.Tensor, k: int, idx: torch.Tensor, stream=None) -> torch.Tensor:
    """TopK of X[b][j]^2 per row of X [B, K] (or [B, 1, K]: one token per unit),
    ascending, into idx (int32, B*k)."""
    if X.dim() == 3:
        if X.shape[1] != 1:
            raise ValueError("X must hold one token per unit")
        X = X[:, 0, :]
    if X.dim() != 2 or X.stride(1) != 1:
        raise ValueError("X must be [B, K] with contiguous rows")
    B, K = X.shape
    d = _dev(X, idx)
    if idx.dtype != torch.int32 or not idx.is_contiguous() or idx.numel() != B * k:
        raise ValueError("idx must be contiguous int32 with B*k elements")
    _check("rmm_select_tokens", lib.rmm_select_tokens(
        X.data_ptr(), _dtype_code(X), B, K, X.stride(0), int(k), idx.data_ptr(), _stream(d, stream)))
    return idx


def rmm_gemv_workspace_size(B: int, M: int, N: int, k: int) -> int:
    return int(lib.rmm_gemv_workspace_size(int(B), int(M), int(N), int(k)))


def rmm_reduced_gemv(X: torch.Tensor, W: torch.Tensor, idx: torch.Tensor, Y: torch.Tensor,
                     workspace: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Decode-step form of rmm_reduced_gemm (M <= 8 rows per unit, bf16):
    Y[b] = X[b][:, I_b] @ W[I_b, :]; `workspace` (uint8,
    rmm_gemv_workspace_size(B, M, N, k) bytes) is allocated here when not given."""
    B, M, K, ldx = _rows(X, "X")
    d = _dev(X, W, idx, Y)
    if W.dim() != 2 or W.shape[0] != K or W.stride(1) != 1:
        raise ValueError("W must be [K, N] with contiguous rows")
    N, ldw = W.shape[1], W.stride(0)
    By, My, Ny, ldy = _rows(Y, "Y")
    if (By, My, Ny) != (B, M, N):
        raise ValueError("Y must be [B, M, N]")
    if not (X.dtype == W.dtype == Y.dtype):
        raise TypeError("X, W and Y must share one dtype")
    if idx.dtype != torch.int32 or not idx.is_contiguous() or idx.numel() % B:
        raise ValueError("idx must be contiguous int32 [B, k]")
    k = idx.numel() // B
    if workspace is None:
        need = rmm_gemv_workspace_size(B, M, N, k)
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=d)
    ws_bytes = workspace.numel() * workspace.element_size()
    _check("rmm_reduced_gemv", lib.rmm_reduced_gemv(
        X.data_ptr(), W.data_ptr(), idx.data_ptr(), _dtype_code(X), B, M, N, K, k, ldx, ldw,
        Y.data_ptr(), ldy, workspace.data_ptr(), ws_bytes, _stream(d, stream)))
    return Y


def rmm_reduced_gemm_kmajor(Xt: torch.Tensor, W: torch.Tensor, idx: torch.Tensor,
                            Y: torch.Tensor, stream=None) -> torch.Tensor:
    """Y[b] = X[b][:, I_b] @ W[I_b, :] from the K-major copy Xt [B, K, M]."""
    B, K, M, ldxt = _rows(Xt, "Xt")
    d = _dev(Xt, W, idx, Y)
    if W.dim() != 2 or W.shape[0] != K or W.stride(1) != 1:
        raise ValueError("W must be [K, N] with contiguous rows")
    N, ldw = W.shape[1], W.stride(0)
    By, My, Ny, ldy = _rows(Y, "Y")
    if (By, My, Ny) != (B, M, N):
        raise ValueError("Y must be [B, M, N]")
    if not (Xt.dtype == W.dtype == Y.dtype == torch.bfloat16):
        raise TypeError("Xt, W and Y must be bfloat16")
    if idx.dtype != torch.int32 or not idx.is_contiguous() or idx.numel() % B:
        raise ValueError("idx must be contiguous int32 [B, k]")
    k = idx.numel() // B
    _check("rmm_reduced_gemm_kmajor", lib.rmm_reduced_gemm_kmajor(
        Xt.data_ptr(), W.data_ptr(), idx.data_ptr(), B, M, N, K, k, ldxt, ldw, Y.data_ptr(),
        ldy, _stream(d, stream)))
    return Y


def swiglu_weight_layout(Wg: torch.Tensor, Wu: torch.Tensor) -> torch.Tensor:
    """The gate and up weights [K, F] as rmm_reduced_gemm_swiglu_kmajor reads
    them: [K, 2F] in 128-column blocks, gate then up of the same 128 channels
    (a column permutation, made once at load time)."""
    if Wg.shape != Wu.shape or Wg.dim() != 2 or Wg.shape[1] % 128:
        raise ValueError("Wg and Wu must be [K, F] with F a multiple of 128")
    K, F = Wg.shape
    return torch.stack([Wg.reshape(K, F // 128, 128), Wu.reshape(K, F // 128, 128)],
                       dim=2).reshape(K, 2 * F).contiguous()


def rmm_gemm_swiglu_workspace_size(B: int, M: int, F: int) -> int:
    return int(lib.rmm_gemm_swiglu_workspace_size(B, M, F))


def rmm_reduced_gemm_swiglu_kmajor(Xt: torch.Tensor, Wgu: torch.Tensor, idx: torch.Tensor,
                                   Ht: torch.Tensor, energy: torch.Tensor,
                                   workspace: torch.Tensor | None = None,
                                   stream=None) -> torch.Tensor:
    """The reduced gate|up product from the K-major copy Xt [B, K, M] with the
    SwiGLU epilogue: writes the down projection's K-major input Ht [B, F, M]
    (rows of stride ldht >= M) and its column energies energy float64 [B, F].
    Wgu [K, 2F] in the layout of swiglu_weight_layout; idx [B, k]."""
    B, K, M, ldxt = _rows(Xt, "Xt")
    if Ht.dim() == 2:
        Ht = Ht.unsqueeze(0)
    if energy.dim() == 1:
        energy = energy.unsqueeze(0)
    d = _dev(Xt, Wgu, idx, Ht, energy)
    if Wgu.dim() != 2 or Wgu.shape[0] != K or Wgu.stride(1) != 1 or Wgu.shape[1] % 2:
        raise ValueError("Wgu must be [K, 2F] with contiguous rows")
    F, ldw = Wgu.shape[1] // 2, Wgu.stride(0)
    if Ht.shape[0] != B or Ht.shape[1] != F or Ht.shape[2] != M:
        raise ValueError("Ht must be [B, F, M]")
    if Ht.stride(2) != 1 or (B > 1 and Ht.stride(0) != F * Ht.stride(1)):
        raise ValueError("Ht rows must be contiguous, with one row stride ldht")
    if tuple(energy.shape) != (B, F) or not energy.is_contiguous() or energy.dtype != torch.float64:
        raise ValueError("energy must be contiguous float64 [B, F]")
    if not (Xt.dtype == Wgu.dtype == Ht.dtype == torch.bfloat16):
        raise TypeError("Xt, Wgu and Ht must be bfloat16")
    if idx.dtype != torch.int32 or not idx.is_contiguous() or idx.numel() % B:
        raise ValueError("idx must be contiguous int32 [B, k]")
    k = idx.numel() // B
    if workspace is None:
        workspace = torch.empty(max(rmm_gemm_swiglu_workspace_size(B, M, F), 1),
                                dtype=torch.uint8, device=d)
    ws_bytes = workspace.numel() * workspace.element_size()
    _check("rmm_reduced_gemm_swiglu_kmajor", lib.rmm_reduced_gemm_swiglu_kmajor(
        Xt.data_ptr(), Wgu.data_ptr(), idx.data_ptr(), B, M, F, K, k, ldxt, ldw, Ht.data_ptr(),
        Ht.stride(1), energy.data_ptr(), workspace.data_ptr(), ws_bytes, _stream(d, stream)))
    return Ht


def rmm_reduced_qk(Q: torch.Tensor, Kc: torch.Tensor, idx: torch.Tensor, S: torch.Tensor,
                   causal: bool = True, scale: float | None = None, stream=None) -> torch.Tensor:
    """Reduced scores for Q [batch, H, Lq, D], Kc [batch, Hkv, Lk, D], idx [batch, H, k]."""
    if Q.dim() == 3:
        Q, Kc, S = Q.unsqueeze(0), Kc.unsqueeze(0), S.unsqueeze(0)
    batch, H, Lq, D = Q.shape
    bk, Hkv, Lk, Dk = Kc.shape
    d = _dev(Q, Kc, idx, S)
    if bk != batch or Dk != D:
        raise ValueError("Kc must be [batch, Hkv, Lk, D]")
    if tuple(S.shape) != (batch, H, Lq, Lk):
        raise ValueError("S must be [batch, H, Lq, Lk]")
    for t, n in ((Q, "Q"), (Kc, "Kc"), (S, "S"), (idx, "idx")):
        if not t.is_contiguous():
            raise ValueError(f"{n} must be contiguous")
    if not (Q.dtype == Kc.dtype == S.dtype):
        raise TypeError("Q, Kc and S must share one dtype")
    if idx.dtype != torch.int32 or idx.numel() % (batch * H):
        raise ValueError("idx must be int32 [batch, H, k]")
    k = idx.numel() // (batch * H)
    if scale is None:
        scale = D ** -0.5
    _check("rmm_reduced_qk", lib.rmm_reduced_qk(
        Q.data_ptr(), Kc.data_ptr(), idx.data_ptr(), _dtype_code(Q), batch, H, Hkv, Lq, Lk, D,
        k, float(scale), 1 if causal else 0, S.data_ptr(), _stream(d, stream)))
    return S


def rmm_reduced_qk_rowstats(Q: torch.Tensor, Kc: torch.Tensor, idx: torch.Tensor, S: torch.Tensor,
                            row_max: torch.Tensor, row_rinv: torch.Tensor, causal: bool = True,
                            scale: float | None = None, stream=None) -> torch.Tensor:
    """rmm_reduced_qk (bf16) that also writes each score row's softmax
    statistics: row_max and row_rinv, float32 [batch*H*Lq]."""
    if Q.dim() != 4 or Kc.dim() != 4 or S.dim() != 4:
        raise ValueError("Q, Kc and S must be 4-D")
    batch, H, Lq, D = Q.shape
    bk, Hkv, Lk, Dk = Kc.shape
    d = _dev(Q, Kc, idx, S, row_max, row_rinv)
    if bk != batch or Dk != D or tuple(S.shape) != (batch, H, Lq, Lk):
        raise ValueError("shapes: Q [b, H, Lq, D], Kc [b, Hkv, Lk, D], S [b, H, Lq, Lk]")
    for t, n in ((Q, "Q"), (Kc, "Kc"), (S, "S"), (idx, "idx")):
        if not t.is_contiguous():
            raise ValueError(f"{n} must be contiguous")
    if not (Q.dtype == Kc.dtype == S.dtype == torch.bfloat16):
        raise TypeError("Q, Kc and S must be bfloat16")
    for t, n in ((row_max, "row_max"), (row_rinv, "row_rinv")):
        if t.dtype != torch.float32 or t.numel() != batch * H * Lq or not t.is_contiguous():
            raise ValueError(f"{n} must be contiguous float32 [batch*H*Lq]")
    if idx.dtype != torch.int32 or idx.numel() % (batch * H):
        raise ValueError("idx must be int32 [batch, H, k]")
    k = idx.numel() // (batch * H)
    if scale is None:
        scale = D ** -0.5
    _check("rmm_reduced_qk_rowstats", lib.rmm_reduced_qk_rowstats(
        Q.data_ptr(), Kc.data_ptr(), idx.data_ptr(), batch, H, Hkv, Lq, Lk, D, k, float(scale),
        1 if causal else 0, S.data_ptr(), row_max.data_ptr(), row_rinv.data_ptr(), _stream(d, stream)))
    return S


def rmm_reduced_attention(Q: torch.Tensor, Kc: torch.Tensor, V: torch.Tensor, idx: torch.Tensor,
                          O: torch.Tensor, causal: bool = True, scale: float | None = None,
                          workspace: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """softmax(reduced scores + mask) V for Q [batch, H, Lq, D], Kc and V
    [batch, Hkv, Lk, D], idx [batch, H, k]; writes O [batch, H, Lq, D].
    `workspace` (uint8, rmm_workspace_size(RMM_OP_ATTENTION, batch*H, Lk, D, k)
    bytes) is allocated here when not given."""
    if Q.dim() == 3:
        Q, Kc, V, O = Q.unsqueeze(0), Kc.unsqueeze(0), V.unsqueeze(0), O.unsqueeze(0)
    batch, H, Lq, D = Q.shape
    bk, Hkv, Lk, Dk = Kc.shape
    d = _dev(Q, Kc, V, idx, O)
    if bk != batch or Dk != D:
        raise ValueError("Kc must be [batch, Hkv, Lk, D]")
    if tuple(V.shape) != (batch, Hkv, Lk, D):
        raise ValueError("V must be [batch, Hkv, Lk, D]")
    if tuple(O.shape) != (batch, H, Lq, D):
        raise ValueError("O must be [batch, H, Lq, D]")
    for t, n in ((Q, "Q"), (Kc, "Kc"), (V, "V"), (O, "O"), (idx, "idx")):
        if not t.is_contiguous():
            raise ValueError(f"{n} must be contiguous")
    if not (Q.dtype == Kc.dtype == V.dtype == O.dtype):
        raise TypeError("Q, Kc, V and O must share one dtype")
    if idx.dtype != torch.int32 or idx.numel() % (batch * H):
        raise ValueError("idx must be int32 [batch, H, k]")
    k = idx.numel() // (batch * H)
    if scale is None:
        scale = D ** -0.5
    if workspace is None:
        workspace = torch.empty(max(rmm_workspace_size(RMM_OP_ATTENTION, batch * H, Lk, D, k), 1),
                                dtype=torch.uint8, device=d)
    ws_bytes = workspace.numel() * workspace.element_size()
    _check("rmm_reduced_attention", lib.rmm_reduced_attention(
        Q.data_ptr(), Kc.data_ptr(), V.data_ptr(), idx.data_ptr(), _dtype_code(Q), batch, H, Hkv,
        Lq, Lk, D, k, float(scale), 1 if causal else 0, O.data_ptr(), workspace.data_ptr(),
        ws_bytes, _stream(d, stream)))
    return O


def rmm_attention_kmajor_workspace_size(batch: int, H: int, Lq: int, Lk: int, D: int,
                                        k: int) -> int:
    return int(lib.rmm_attention_kmajor_workspace_size(batch, H, Lq, Lk, D, k))


def rmm_reduced_attention_kmajor(Q: torch.Tensor, Kc: torch.Tensor, V: torch.Tensor,
                                 idx: torch.Tensor, Ot: torch.Tensor, energy: torch.Tensor,
                                 causal: bool = True, scale: float | None = None,
                                 workspace: torch.Tensor | None = None,
                                 stream=None) -> torch.Tensor:
    """The reduced attention block of rmm_reduced_attention, written as the
    output projection's K-major input Ot [batch, H*D, ldot] (a view whose
    rows have stride ldot >= Lq) with that input's column energies
    energy float64 [batch, H*D].  `workspace` (uint8,
    rmm_attention_kmajor_workspace_size(...) bytes, 256-byte aligned) is
    allocated here when not given."""
    if Q.dim() == 3:
        Q, Kc, V = Q.unsqueeze(0), Kc.unsqueeze(0), V.unsqueeze(0)
    if Ot.dim() == 2:
        Ot = Ot.unsqueeze(0)
    if energy.dim() == 1:
        energy = energy.unsqueeze(0)
    batch, H, Lq, D = Q.shape
    bk, Hkv, Lk, Dk = Kc.shape
    d = _dev(Q, Kc, V, idx, Ot, energy)
    if bk != batch or Dk != D:
        raise ValueError("Kc must be [batch, Hkv, Lk, D]")
    if tuple(V.shape) != (batch, Hkv, Lk, D):
        raise ValueError("V must be [batch, Hkv, Lk, D]")
    if Ot.shape[0] != batch or Ot.shape[1] != H * D or Ot.shape[2] < Lq:
        raise ValueError("Ot must be [batch, H*D, >= Lq]")
    if Ot.stride(2) != 1 or Ot.stride(0) != Ot.shape[1] * Ot.stride(1):
        raise ValueError("Ot rows must be contiguous, with one row stride ldot")
    if tuple(energy.shape) != (batch, H * D) or not energy.is_contiguous() or \
            energy.dtype != torch.float64:
        raise ValueError("energy must be contiguous float64 [batch, H*D]")
    for t, n in ((Q, "Q"), (Kc, "Kc"), (V, "V"), (idx, "idx")):
        if not t.is_contiguous():
            raise ValueError(f"{n} must be contiguous")
    if not (Q.dtype == Kc.dtype == V.dtype == Ot.dtype):
        raise TypeError("Q, Kc, V and Ot must share one dtype")
    if idx.dtype != torch.int32 or idx.numel() % (batch * H):
        raise ValueError("idx must be int32 [batch, H, k]")
    k = idx.numel() // (batch * H)
    if scale is None:
        scale = D ** -0.5
    if workspace is None:
        workspace = torch.empty(max(rmm_attention_kmajor_workspace_size(batch, H, Lq, Lk, D, k), 1),
                                dtype=torch.uint8, device=d)
    ws_bytes = workspace.numel() * workspace.element_size()
    _check("rmm_reduced_attention_kmajor", lib.rmm_reduced_attention_kmajor(
        Q.data_ptr(), Kc.data_ptr(), V.data_ptr(), idx.data_ptr(), _dtype_code(Q), batch, H, Hkv,
        Lq, Lk, D, k, float(scale), 1 if causal else 0, Ot.data_ptr(), Ot.stride(1),
        energy.data_ptr(), workspace.data_ptr(), ws_bytes, _stream(d, stream)))
    return Ot


def rmm_reduced_pv(P: torch.Tensor, V: torch.Tensor, kt: int, O: torch.Tensor,
                   idx_out: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
                   stream=None) -> torch.Tensor:
    """Token-axis reduced value product (Sec. 3.3): per query head u, the kt
    tokens with the largest column norms of P[u] and O[u] = P[u][:, T] @
    V[kv(u)][T, :].  P: [batch, H, Lq, Lk] (rows contiguous, any row stride),
    V: [batch, Hkv, Lk, D] contiguous, O: [batch, H, Lq, D] contiguous;
    `idx_out` (int32 [batch*H*kt]) receives the token sets when given."""
    if P.dim() != 4 or V.dim() != 4 or O.dim() != 4:
        raise ValueError("P, V and O must be 4-D")
    batch, H, Lq, Lk = P.shape
    if P.stride(3) != 1 or P.stride(1) != Lq * P.stride(2) or P.stride(0) != H * P.stride(1):
        raise ValueError("P must be [batch, H, Lq, Lk] with contiguous rows and packed rows")
    ldp = P.stride(2)
    if V.shape[0] != batch or V.shape[2] != Lk or not V.is_contiguous():
        raise ValueError("V must be contiguous [batch, Hkv, Lk, D]")
    Hkv, D = V.shape[1], V.shape[3]
    if tuple(O.shape) != (batch, H, Lq, D) or not O.is_contiguous():
        raise ValueError("O must be contiguous [batch, H, Lq, D]")
    d = _dev(P, V, O)
    if not (P.dtype == V.dtype == O.dtype):
        raise TypeError("P, V and O must share one dtype")
    if idx_out is not None and (idx_out.dtype != torch.int32 or idx_out.numel() != batch * H * kt
                                or not idx_out.is_contiguous()):
        raise ValueError("idx_out must be contiguous int32 [batch*H*kt]")
    if workspace is None:
        workspace = torch.empty(max(rmm_workspace_size(RMM_OP_PV, batch * H, Lq, Lk, kt), 1),
                                dtype=torch.uint8, device=d)
    ws_bytes = workspace.numel() * workspace.element_size()
    _check("rmm_reduced_pv", lib.rmm_reduced_pv(
        P.data_ptr(), V.data_ptr(), _dtype_code(P), batch, H, Hkv, Lq, Lk, D, ldp, int(kt),
        O.data_ptr(), _ptr(idx_out), workspace.data_ptr(), ws_bytes, _stream(d, stream)))
    return O


def rmm_linear(X: torch.Tensor, W: torch.Tensor, r: float, Y: torch.Tensor,
               idx_out: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
               stream=None) -> torch.Tensor:
    """Fused score -> select -> gathered GEMM at retention ratio r."""
    B, M, K, ldx = _rows(X, "X")
    d = _dev(X, W, Y)
    if W.dim() != 2 or W.shape[0] != K or W.stride(1) != 1:
        raise ValueError("W must be [K, N] with contiguous rows")
    N, ldw = W.shape[1], W.stride(0)
    By, My, Ny, ldy = _rows(Y, "Y")
    if (By, My, Ny) != (B, M, N):
        raise ValueError("Y must be [B, M, N]")
    if not (X.dtype == W.dtype == Y.dtype):
        raise TypeError("X, W and Y must share one dtype")
    k = rmm_retained_count(r, K)
    if idx_out is not None and (idx_out.dtype != torch.int32 or idx_out.numel() != B * max(k, 0)
                                or not idx_out.is_contiguous()):
        raise ValueError("idx_out must be contiguous int32 [B, k]")
    if workspace is None:
        workspace = torch.empty(max(rmm_workspace_size(RMM_OP_LINEAR, B, M, K, k), 1),
                                dtype=torch.uint8, device=d)
    ws_bytes = workspace.numel() * workspace.element_size()
    _check("rmm_linear", lib.rmm_linear(
        X.data_ptr(), W.data_ptr(), float(r), _dtype_code(X), B, M, N, K, ldx, ldw,
        Y.data_ptr(), ldy, _ptr(idx_out), workspace.data_ptr(), ws_bytes, _stream(d, stream)))
    return Y


def rmm_noalloc_scratch_bytes() -> int:
    return int(lib.rmm_noalloc_scratch_bytes())


def rmm_linear_noalloc(X: torch.Tensor, W: torch.Tensor, r: float, Y: torch.Tensor,
                       idx_out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """rmm_linear with the library's fixed scratch instead of a workspace:
    neither this wrapper nor the call allocates device memory (usable under
    HIP graph capture).  Calls that overlap in time on one GPU race."""
    B, M, K, ldx = _rows(X, "X")
    d = _dev(X, W, Y)
    if W.dim() != 2 or W.shape[0] != K or W.stride(1) != 1:
        raise ValueError("W must be [K, N] with contiguous rows")
    N, ldw = W.shape[1], W.stride(0)
    By, My, Ny, ldy = _rows(Y, "Y")
    if (By, My, Ny) != (B, M, N):
        raise ValueError("Y must be [B, M, N]")
    if not (X.dtype == W.dtype == Y.dtype):
        raise TypeError("X, W and Y must share one dtype")
    k = rmm_retained_count(r, K)
    if idx_out is not None and (idx_out.dtype != torch.int32 or idx_out.numel() != B * max(k, 0)
                                or not idx_out.is_contiguous()):
        raise ValueError("idx_out must be contiguous int32 [B, k]")
    _check("rmm_linear_noalloc", lib.rmm_linear_noalloc(
        X.data_ptr(), W.data_ptr(), float(r), _dtype_code(X), B, M, N, K, ldx, ldw,
        Y.data_ptr(), ldy, _ptr(idx_out), _stream(d, stream)))
    return Y


def rmm_rmsnorm_kmajor_workspace_size(B: int, M: int, K: int) -> int:
    return int(lib.rmm_rmsnorm_kmajor_workspace_size(int(B), int(M), int(K)))


def rmm_rmsnorm_kmajor(X: torch.Tensor, gamma: torch.Tensor, eps: float, Xt: torch.Tensor,
                       energy: torch.Tensor, workspace: torch.Tensor | None = None,
                       stream=None) -> torch.Tensor:
    """RMSNorm of X [B, M, K] (or [M, K]) with weight gamma [K], written
    K-major into Xt [B, K, M] (row stride Xt.stride(-2)) with the column
    energies of the normalised rows in energy (float64 [B*K])."""
    B, M, K, ldx = _rows(X, "X")
    d = _dev(X, gamma, Xt, energy)
    Bt, Kt, Mt, ldxt = _rows(Xt, "Xt")
    if (Bt, Kt, Mt) != (B, K, M):
        raise ValueError("Xt must be [B, K, M]")
    if gamma.numel() != K or not gamma.is_contiguous():
        raise ValueError("gamma must be a contiguous [K] tensor")
    if not (X.dtype == gamma.dtype == Xt.dtype == torch.bfloat16):
        raise TypeError("X, gamma and Xt must be bfloat16")
    if energy.dtype != torch.float64 or energy.numel() != B * K or not energy.is_contiguous():
        raise ValueError("energy must be contiguous float64 [B*K]")
    if workspace is None:
        workspace = torch.empty(max(rmm_rmsnorm_kmajor_workspace_size(B, M, K), 1),
                                dtype=torch.uint8, device=d)
    ws_bytes = workspace.numel() * workspace.element_size()
    _check("rmm_rmsnorm_kmajor", lib.rmm_rmsnorm_kmajor(
        X.data_ptr(), gamma.data_ptr(), float(eps), B, M, K, ldx, Xt.data_ptr(), ldxt,
        energy.data_ptr(), workspace.data_ptr(), ws_bytes, _stream(d, stream)))
    return Xt


def rmm_attention_weights_kmajor_workspace_size(batch: int, H: int, Lq: int, Lk: int) -> int:
    return int(lib.rmm_attention_weights_kmajor_workspace_size(batch, H, Lq, Lk))


def rmm_attention_weights_kmajor(S: torch.Tensor, Pt: torch.Tensor, energy: torch.Tensor,
                                 causal: bool = True, workspace: torch.Tensor | None = None,
                                 stream=None, row_max: torch.Tensor | None = None,
                                 row_rinv: torch.Tensor | None = None) -> torch.Tensor:
    """Softmax weights of the scores S [batch, H, Lq, Lk] written K-major into
    Pt [batch, H, Lk, Lq] (row stride Pt.stride(-2)), with their token
    energies (float64 [batch*H*Lk]).  With row_max and row_rinv (float32
    [batch*H*Lq], e.g. from rmm_reduced_qk_rowstats) the weights use those
    row statistics (rmm_attention_weights_kmajor_rowstats)."""
    if S.dim() != 4 or Pt.dim() != 4:
        raise ValueError("S and Pt must be 4-D")
    batch, H, Lq, Lk = S.shape
    d = _dev(S, Pt, energy)
    if tuple(Pt.shape) != (batch, H, Lk, Lq):
        raise ValueError("Pt must be [batch, H, Lk, Lq]")
    if S.stride(3) != 1 or S.stride(1) != Lq * S.stride(2) or S.stride(0) != H * Lq * S.stride(2):
        raise ValueError("S rows must be contiguous and its heads packed")
    if Pt.stride(3) != 1 or Pt.stride(1) != Lk * Pt.stride(2) or Pt.stride(0) != H * Lk * Pt.stride(2):
        raise ValueError("Pt rows must be contiguous and its heads packed")
    if not (S.dtype == Pt.dtype == torch.bfloat16):
        raise TypeError("S and Pt must be bfloat16")
    if energy.dtype != torch.float64 or energy.numel() != batch * H * Lk or not energy.is_contiguous():
        raise ValueError("energy must be contiguous float64 [batch*H*Lk]")
    if workspace is None:
        workspace = torch.empty(max(rmm_attention_weights_kmajor_workspace_size(batch, H, Lq, Lk), 1),
                                dtype=torch.uint8, device=d)
    ws_bytes = workspace.numel() * workspace.element_size()
    if (row_max is None) != (row_rinv is None):
        raise ValueError("give both row_max and row_rinv, or neither")
    if row_max is None:
        _check("rmm_attention_weights_kmajor", lib.rmm_attention_weights_kmajor(
            S.data_ptr(), batch, H, Lq, Lk, S.stride(2), 1 if causal else 0, Pt.data_ptr(),
            Pt.stride(2), energy.data_ptr(), workspace.data_ptr(), ws_bytes, _stream(d, stream)))
        return Pt
    _dev(S, row_max, row_rinv)
    for t, n in ((row_max, "row_max"), (row_rinv, "row_rinv")):
        if t.dtype != torch.float32 or t.numel() != batch * H * Lq or not t.is_contiguous():
            raise ValueError(f"{n} must be contiguous float32 [batch*H*Lq]")
    _check("rmm_attention_weights_kmajor_rowstats", lib.rmm_attention_weights_kmajor_rowstats(
        S.data_ptr(), batch, H, Lq, Lk, S.stride(2), 1 if causal else 0, row_max.data_ptr(),
        row_rinv.data_ptr(), Pt.data_ptr(), Pt.stride(2), energy.data_ptr(), workspace.data_ptr(),
        ws_bytes, _stream(d, stream)))
    return Pt


def rmm_reduced_pv_kmajor(Pt: torch.Tensor, V: torch.Tensor, idx: torch.Tensor, O: torch.Tensor,
                          causal: bool = True, stream=None) -> torch.Tensor:
    """O[b, h] = Pt[b, h][T, :]^T V[b, h // (H/Hkv)][T, :] with the token sets
    idx [batch*H, kt] (ascending)."""
    if Pt.dim() != 4 or V.dim() != 4 or O.dim() != 4:
        raise ValueError("Pt, V and O must be 4-D")
    batch, H, Lk, Lq = Pt.shape
    _, Hkv, Lkv, D = V.shape
    d = _dev(Pt, V, idx, O)
    if Lkv != Lk or tuple(O.shape) != (batch, H, Lq, D) or H % Hkv:
        raise ValueError("shapes: Pt [b, H, Lk, Lq], V [b, Hkv, Lk, D], O [b, H, Lq, D]")
    if Pt.stride(3) != 1 or Pt.stride(1) != Lk * Pt.stride(2) or Pt.stride(0) != H * Lk * Pt.stride(2):
        raise ValueError("Pt rows must be contiguous and its heads packed")
    if not (V.is_contiguous() and O.is_contiguous()):
        raise ValueError("V and O must be contiguous")
    if not (Pt.dtype == V.dtype == O.dtype == torch.bfloat16):
        raise TypeError("Pt, V and O must be bfloat16")
    if idx.dtype != torch.int32 or not idx.is_contiguous() or idx.numel() % (batch * H):
        raise ValueError("idx must be contiguous int32 [batch*H, kt]")
    kt = idx.numel() // (batch * H)
    _check("rmm_reduced_pv_kmajor", lib.rmm_reduced_pv_kmajor(
        Pt.data_ptr(), V.data_ptr(), idx.data_ptr(), batch, H, Hkv, Lq, Lk, D, kt, Pt.stride(2),
        1 if causal else 0, O.data_ptr(), _stream(d, stream)))
    return O


def _decode_groups(groups):
    """[(X [B, K], W [K, N], k, idx [B*k] int32, Y [B, N])] -> ctypes array, B."""
    arr = (DecodeGroup * len(groups))()
    B = None
    for i, (X, W, k, idx, Y) in enumerate(groups):
        if X.dim() != 2 or W.dim() != 2 or Y.dim() != 2:
            raise ValueError("X [B, K], W [K, N] and Y [B, N] must be 2-D")
        if B is None:
            B = X.shape[0]
        if X.shape[0] != B or Y.shape[0] != B or W.shape[0] != X.shape[1] or Y.shape[1] != W.shape[1]:
            raise ValueError("group shapes disagree: X [B, K], W [K, N], Y [B, N]")
        if X.stride(1) != 1 or W.stride(1) != 1 or Y.stride(1) != 1:
            raise ValueError("rows must be contiguous")
        if not (X.dtype == W.dtype == Y.dtype == torch.bfloat16):
            raise TypeError("X, W and Y must be bfloat16")
        if idx.dtype != torch.int32 or idx.numel() != B * k or not idx.is_contiguous():
            raise ValueError("idx must be contiguous int32 [B*k]")
        _dev(X, W, idx, Y)
        arr[i] = DecodeGroup(X.data_ptr(), W.data_ptr(), idx.data_ptr(), Y.data_ptr(), X.shape[1],
                             W.shape[1], int(k), X.stride(0), W.stride(0), Y.stride(0))
    return arr, B


def rmm_decode_step_workspace_size(groups) -> int:
    arr, B = _decode_groups(groups)
    return int(lib.rmm_decode_step_workspace_size(arr, len(groups), B))


def rmm_decode_products(groups, workspace: torch.Tensor | None = None, stream=None):
    """For each group (X [B, K], W [K, N], k, idx [B*k], Y [B, N]) with idx
    holding caller-made ascending sets: Y = the reduced product; all groups
    in two launches (rmm_decode_step without its selection)."""
    arr, B = _decode_groups(groups)
    d = groups[0][0].device
    need = int(lib.rmm_decode_step_workspace_size(arr, len(groups), B))
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=d)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check("rmm_decode_products", lib.rmm_decode_products(arr, len(groups), B, _ptr(workspace),
                                                          ws_bytes, _stream(d, stream)))


def rmm_decode_products_shared_workspace_size(groups) -> int:
    arr, B = _decode_groups(groups)
    return int(lib.rmm_decode_products_shared_workspace_size(arr, len(groups), B))


def rmm_decode_products_shared(groups, workspace: torch.Tensor | None = None, stream=None):
    """The same products as rmm_decode_products (B <= 32 sequences), reading
    each weight row that some sequence keeps once for the whole batch; equal
    to it within rounding."""
    arr, B = _decode_groups(groups)
    d = groups[0][0].device
    if workspace is None:
        need = int(lib.rmm_decode_products_shared_workspace_size(arr, len(groups), B))
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=d)
    ws_bytes = workspace.numel() * workspace.element_size()
    _check("rmm_decode_products_shared",
           lib.rmm_decode_products_shared(arr, len(groups), B, _ptr(workspace), ws_bytes,
                                          _stream(d, stream)))


def rmm_decode_step_shared(groups, workspace: torch.Tensor | None = None, stream=None):
    """For each group (X [B, K], W [K, N], k, idx [B*k], Y [B, N]), B <= 32:
    idx = each token's TopK (as rmm_decode_step), Y = the shared-rows
    products over those sets (rmm_decode_products_shared)."""
    arr, B = _decode_groups(groups)
    d = groups[0][0].device
    if workspace is None:
        need = int(lib.rmm_decode_products_shared_workspace_size(arr, len(groups), B))
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=d)
    ws_bytes = workspace.numel() * workspace.element_size()
    _check("rmm_decode_step_shared",
           lib.rmm_decode_step_shared(arr, len(groups), B, _ptr(workspace), ws_bytes, _stream(d, stream)))


def rmm_decode_step(groups, workspace: torch.Tensor | None = None, stream=None):
    """For each group (X [B, K], W [K, N], k, idx [B*k], Y [B, N]): idx = the
    TopK of each token's squared activations, Y = the reduced product; all
    groups in three launches."""
    arr, B = _decode_groups(groups)
    d = groups[0][0].device
    need = int(lib.rmm_decode_step_workspace_size(arr, len(groups), B))
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=d)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check("rmm_decode_step", lib.rmm_decode_step(arr, len(groups), B, _ptr(workspace), ws_bytes,
                                                  _stream(d, stream)))
