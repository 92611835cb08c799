"""Seeded synthetic inputs for the RMM hot path.

This module is shared by the oracle tests, the GPU parity tests and the
benchmark.  It holds no part of RMM's arithmetic (no scoring, no selection,
no products): it only draws random tensors with the shapes and value
distributions of the workloads below and encodes them as bf16 or fp32 bytes.
Both the oracle and the HIP path consume the same bytes.

Value recipe (the paper's models are replaced by synthetic tensors of their
layer shapes; the paper runs in bf16, Appendix A "Hardware and framework"):

* activations: i.i.d. N(0, 1), with a fixed set of "outlier" channels
  (columns of the activation matrix) multiplied by a constant;
* weights: i.i.d. N(0, 0.02^2) (0.02 read as the standard deviation);
* attention Q/K with per-head heavy-tailed dimensions: entry
  ``c[h, j] * z`` with ``z ~ N(0, 1)`` and ``c[h, j] = |t_3|`` drawn once per
  (head, dimension), independently for Q and K.

Every tensor gets its own PCG64 stream ``default_rng([seed, tensor_id])`` so
that adding a tensor never changes another.  bf16 values come from fp32
samples by round-to-nearest-even.
"""
from __future__ import annotations

from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
import os

import numpy as np

__all__ = [
    "f32_to_bf16_bits", "bf16_bits_to_f32", "Projection", "AttentionShape",
    "Workload", "WORKLOADS", "rng_for", "activation", "weight",
    "heavy_tailed_heads", "outlier_heads", "encode", "decode",
    "attention_score_bits",
]


_POOL = ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1))


# ---------------------------------------------------------------------------
# bf16 encoding (storage format only)
# ---------------------------------------------------------------------------

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16) by round-to-nearest-even.

    NaN inputs map to a quiet NaN; infinities stay infinities.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, dtype=np.uint16)
    xf, of = x.reshape(-1), out.reshape(-1)

    def part(lo_hi):
        lo, hi = lo_hi
        u = xf[lo:hi].view(np.uint32)
        # no uint32 overflow: the largest non-NaN pattern is -inf (0xff800000)
        r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
        o = r.astype(np.uint16)
        nan = np.isnan(xf[lo:hi])
        if nan.any():
            o[nan] = ((u[nan] >> np.uint32(16)) | np.uint32(0x0040)).astype(np.uint16)
        of[lo:hi] = o

    n, step = xf.shape[0], 1 << 22
    list(_POOL.map(part, [(i, min(n, i + step)) for i in range(0, n, step)]))
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> exact fp32 values."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def encode(x_f32: np.ndarray, dtype: str) -> np.ndarray:
    """Storage bytes for a tensor: uint16 bf16 bits, or fp32 as is."""
    if dtype == "bf16":
        return f32_to_bf16_bits(x_f32)
    if dtype == "f32":
        return np.ascontiguousarray(x_f32, dtype=np.float32)
    raise ValueError(f"unknown dtype {dtype!r}")


def decode(stored: np.ndarray, dtype: str) -> np.ndarray:
    """Exact fp32 values of stored bytes (bf16 bits or fp32)."""
    if dtype == "bf16":
        return bf16_bits_to_f32(stored)
    if dtype == "f32":
        return np.asarray(stored, dtype=np.float32)
    raise ValueError(f"unknown dtype {dtype!r}")


# ---------------------------------------------------------------------------
# generators
# ---------------------------------------------------------------------------

def rng_for(seed: int, tensor_id: int) -> np.random.Generator:
    """Independent PCG64 stream per (seed, tensor id)."""
    return np.random.Generator(np.random.PCG64([seed, tensor_id]))


_BLOCK_ROWS = 64


def normal_blocks(key, shape) -> np.ndarray:
    """N(0,1) float32 array of ``shape`` (at least 2-D: [..., rows, cols]).

    Rows are drawn in fixed blocks of 64, each from its own PCG64 stream
    keyed by (key, leading index, block), in parallel threads.  A draw with
    fewer rows is therefore exactly the leading rows of a longer one.
    """
    shape = tuple(int(v) for v in shape)
    out = np.empty(shape, dtype=np.float32)
    lead, R, C = shape[:-2], shape[-2], shape[-1]
    jobs = [(li, b) for li in np.ndindex(*lead) for b in range(-(-R // _BLOCK_ROWS))]

    def fill(job):
        li, b = job
        r0, r1 = b * _BLOCK_ROWS, min(R, (b + 1) * _BLOCK_ROWS)
        g = np.random.Generator(np.random.PCG64([*key, *li, b]))
        out[li + (slice(r0, r1),)] = g.standard_normal(size=(r1 - r0, C), dtype=np.float32)

    list(_POOL.map(fill, jobs))
    return out


def activation(key, shape, n_outlier: int, outlier_scale: float) -> np.ndarray:
    """N(0,1) activations [..., M, K] with ``n_outlier`` channels scaled.

    ``key`` = (seed, tensor id).  The outlier channels are the same for every
    row (they are channels of the hidden state, i.e. columns of the
    activation matrix), chosen from the stream of ``key``.
    """
    K = shape[-1]
    x = normal_blocks(key, shape)
    if n_outlier > 0:
        cols = rng_for(*key).choice(K, size=n_outlier, replace=False)
        x[..., cols] *= np.float32(outlier_scale)
    return x


def weight(key, K: int, N: int, std: float = 0.02) -> np.ndarray:
    """Weights [K x N] ~ N(0, std^2) (row k = contraction index k)."""
    w = normal_blocks(key, (K, N))
    w *= np.float32(std)
    return w


def heavy_tailed_heads(key, H: int, L: int, D: int, nu: float = 3.0) -> np.ndarray:
    """[H x L x D]: entry c[h,j]*z, z ~ N(0,1), c[h,j] = |Student-t(nu)|."""
    c = np.abs(rng_for(*key).standard_t(nu, size=(H, 1, D))).astype(np.float32)
    z = normal_blocks(key, (H, L, D))
    z *= c
    return z


def outlier_heads(key, H: int, L: int, D: int, frac: float, scale: float) -> np.ndarray:
    """[H x L x D] N(0,1) with ``round(frac*H*D)`` of the H*D channels scaled."""
    z = normal_blocks(key, (H, L, D))
    n_out = int(round(frac * H * D))
    if n_out > 0:
        for c in rng_for(*key).choice(H * D, size=n_out, replace=False):
            z[c // D, :, c % D] *= np.float32(scale)
    return z


_SCORE_ROWS = 256


def _score_block(key, b_h, h: int, r0: int, r1: int, Lq: int, causal: bool,
                 spread: float) -> np.ndarray:
    """Rows r0..r1-1 of head h's synthetic scores (float32), one PCG64 stream
    per (key, head, row block)."""
    g = np.random.Generator(np.random.PCG64([*key, h, r0 // _SCORE_ROWS]))
    s = g.standard_normal(size=(r1 - r0, b_h.shape[0]), dtype=np.float32)
    s *= np.float32(spread)
    s += b_h[None, :]
    if causal:
        Lk = b_h.shape[0]
        t = np.arange(Lk)[None, :]
        i = np.arange(r0, r1)[:, None]
        s[t > i + (Lk - Lq)] = -np.inf
    return s


def attention_score_bits(key, H: int, Lq: int, Lk: int, causal: bool, spread: float = 2.0,
                         nu: float = 3.0, softmax: bool = False) -> np.ndarray:
    """bf16 bits [H x Lq x Lk] of synthetic attention scores, or (with
    ``softmax``) of the attention weights made from them.

    Scores: ``spread * z + b[h, t]`` with z ~ N(0, 1) per entry and a
    per-(head, key) salience ``b = |Student-t(nu)|`` (a few keys draw much of
    every query's weight, as attention sinks do); with ``causal`` the entries
    t > i + (Lk - Lq) are -inf.  Weights: the row softmax of those float32
    scores, computed in float32 (masked entries 0).  Made on the host from
    seeded draws in blocks of 256 rows, each from its own PCG64 stream."""
    b = np.abs(rng_for(*key).standard_t(nu, size=(H, Lk))).astype(np.float32)
    out = np.empty((H, Lq, Lk), dtype=np.uint16)

    def block(job):
        h, r0 = job
        r1 = min(Lq, r0 + _SCORE_ROWS)
        s = _score_block(key, b[h], h, r0, r1, Lq, causal, spread)
        if softmax:
            m = s.max(axis=1, keepdims=True)
            m[~np.isfinite(m)] = 0.0                 # rows with every key masked
            s -= m
            np.exp(s, out=s)
            tot = s.sum(axis=1, keepdims=True)
            tot[tot == 0] = 1.0
            s /= tot
        out[h, r0:r1] = _bits_serial(s)

    list(_POOL.map(block, [(h, r0) for h in range(H) for r0 in range(0, Lq, _SCORE_ROWS)]))
    return out


def _bits_serial(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bits by round-to-nearest-even for finite values and +-inf
    (no NaN handling: the score recipes hold none)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u.astype(np.uint64) + 0x7FFF + ((u >> np.uint32(16)) & np.uint32(1))) >> 16
    return r.astype(np.uint16)


# ---------------------------------------------------------------------------
# workload catalogue
# ---------------------------------------------------------------------------

@dataclass(frozen=True)
class Projection:
    """One projection Y[M x N] = X[M x K] W[K x N] with its own input X."""
    name: str
    input_name: str     # projections with the same input share X
    K: int
    N: int


@dataclass(frozen=True)
class AttentionShape:
    H: int
    Hkv: int
    L: int              # Lq = Lk = L (prefill)
    D: int
    causal: bool = True
    recipe: str = "outlier"   # "outlier" or "heavy_tailed"


@dataclass(frozen=True)
class Workload:
    name: str
    description: str
    dtype: str                       # "f32" or "bf16"
    M: int                           # tokens of the one sequence
    inputs: dict = field(default_factory=dict)   # input name -> (K, n_outlier, scale)
    projections: tuple = ()
    attention: AttentionShape | None = None
    ratios: tuple = (0.25, 0.5, 0.75, 1.0)
    seed: int = 0

    def projection_flops(self, k_of) -> int:
        """2*M*N*k summed over projections, with k = k_of(K)."""
        return sum(2 * self.M * p.N * k_of(p.K) for p in self.projections)


def _pct(K: int, frac: float = 0.01) -> int:
    return int(round(frac * K))


def _llama_layer(name, desc, M, hidden, H, Hkv, D, mlp, seed=0):
    inputs = {
        "attn_in": (hidden, _pct(hidden), 20.0),
        "o_in": (H * D, _pct(H * D), 20.0),
        "mlp_in": (hidden, _pct(hidden), 20.0),
        "down_in": (mlp, _pct(mlp), 20.0),
    }
    projs = (
        Projection("q", "attn_in", hidden, H * D),
        Projection("k", "attn_in", hidden, Hkv * D),
        Projection("v", "attn_in", hidden, Hkv * D),
        Projection("o", "o_in", H * D, hidden),
        Projection("gate", "mlp_in", hidden, mlp),
        Projection("up", "mlp_in", hidden, mlp),
        Projection("down", "down_in", mlp, hidden),
    )
    return Workload(name, desc, "bf16", M, inputs, projs,
                    AttentionShape(H, Hkv, M, D, True, "outlier"), seed=seed)


WORKLOADS = {
    "linear_f32": Workload(
        "linear_f32", "single fp32 linear layer, 128 tokens x 512 -> 512",
        "f32", 128, {"x": (512, 8, 10.0)},
        (Projection("linear", "x", 512, 512),), None, ratios=(0.5, 1.0)),
    "mlp_1b": Workload(
        "mlp_1b", "1B-class gated-MLP projections, 2048 tokens, hidden 2048, MLP 8192",
        "bf16", 2048,
        {"mlp_in": (2048, _pct(2048), 20.0), "down_in": (8192, _pct(8192), 20.0)},
        (Projection("gate", "mlp_in", 2048, 8192),
         Projection("up", "mlp_in", 2048, 8192),
         Projection("down", "down_in", 8192, 2048))),
    "attn_4k": Workload(
        "attn_4k", "attention head-dim reduction, 32 heads x 4096 tokens x 128, causal",
        "bf16", 4096, {}, (), AttentionShape(32, 32, 4096, 128, True, "heavy_tailed")),
    "layer_8b": _llama_layer(
        "layer_8b", "8B-class decoder layer, seq 8192, hidden 4096, 32/8 heads, MLP 14336",
        8192, 4096, 32, 8, 128, 14336),
    "layer_70b": _llama_layer(
        "layer_70b", "70B-class decoder layer, seq 16384, hidden 8192, 64/8 heads, MLP 28672",
        16384, 8192, 64, 8, 128, 28672),
}


# tensor ids: inputs 0..99, weights 100..199, attention Q/K/V 200/201/202
_INPUT_IDS = {"x": 0, "attn_in": 1, "o_in": 2, "mlp_in": 3, "down_in": 4}
_WEIGHT_IDS = {"linear": 100, "q": 101, "k": 102, "v": 103, "o": 104,
               "gate": 105, "up": 106, "down": 107}


def workload_input(wl: Workload, name: str, M: int | None = None) -> np.ndarray:
    """fp32 samples of activation ``name`` [M x K] (before bf16 rounding).

    ``M`` below the workload's token count takes the first M tokens of the
    same draw's distribution (a fresh draw of M rows from the same stream).
    """
    K, n_out, scale = wl.inputs[name]
    return activation((wl.seed, _INPUT_IDS[name]), (wl.M if M is None else M, K), n_out, scale)


def workload_weight(wl: Workload, proj: Projection) -> np.ndarray:
    return weight((wl.seed, _WEIGHT_IDS[proj.name]), proj.K, proj.N)


def workload_qk(wl: Workload, L: int | None = None):
    """fp32 samples of (Q [H x L x D], K [Hkv x L x D])."""
    a = wl.attention
    L = a.L if L is None else L
    kq, kk = (wl.seed, 200), (wl.seed, 201)
    if a.recipe == "heavy_tailed":
        return (heavy_tailed_heads(kq, a.H, L, a.D),
                heavy_tailed_heads(kk, a.Hkv, L, a.D))
    return (outlier_heads(kq, a.H, L, a.D, 0.01, 20.0),
            outlier_heads(kk, a.Hkv, L, a.D, 0.01, 20.0))


def workload_v(wl: Workload, L: int | None = None) -> np.ndarray:
    """fp32 samples of the value rows V [Hkv x L x D], N(0, 1)."""
    a = wl.attention
    L = a.L if L is None else L
    return normal_blocks((wl.seed, 202), (a.Hkv, L, a.D))


def random_case(seed: int, shape, dtype: str, n_outlier: int = 0,
                outlier_scale: float = 10.0, std: float = 1.0) -> np.ndarray:
    """Stored bytes of a generic random tensor for parity/edge-case tests."""
    shape = tuple(shape)
    x = activation((seed, 1000 + len(shape)), shape if len(shape) > 1 else (1,) + shape,
                   n_outlier, outlier_scale).reshape(shape)
    if std != 1.0:
        x *= np.float32(std)
    return encode(x, dtype)


def integer_case(seed: int, shape, lo: int, hi: int, dtype: str) -> np.ndarray:
    """Stored bytes of small integers in [lo, hi] (exact in bf16 and fp32).

    Integer-valued inputs make every sum of squares exact in fp64, so ties
    between energies are exact and the tie rule is exercised bit for bit.
    """
    rng = rng_for(seed, 2000 + len(shape))
    x = rng.integers(lo, hi + 1, size=tuple(shape)).astype(np.float32)
    return encode(x, dtype)


def ceil_div(a: int, b: int) -> int:
    return -(-a // b)

