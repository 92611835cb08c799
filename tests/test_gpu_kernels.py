"""GPU parity of each librmm entry point against the CPU oracle, at sizes the
oracle finishes in seconds that still span several tiles and ragged tails,
plus the edge cases (k = 1, k = K, single rows/columns, ties, NaN/Inf,
unaligned rows, batches of units).  All calls go through the C-ABI."""
import math

import numpy as np
import pytest
import torch

import paper_2608_13426_amd as rmm
import workloads as wl
from oracle import rmm_oracle as ro
from tests.gpu_util import (gpu, require_gpu, to_device, from_device, torch_dtype,
                            check_energies, check_index_sets, check_product,
                            isclose_inf_pattern)

pytestmark = gpu


def _score_ws(B, M, K, dev):
    n = rmm.rmm_workspace_size(rmm.RMM_OP_SCORE, B, M, K)
    return torch.empty(max(n, 1), dtype=torch.uint8, device=dev)


def _energies_gpu(Xd, B, M, K, dev):
    e = torch.empty(B * K, dtype=torch.float64, device=dev)
    rmm.rmm_score(Xd, e, _score_ws(B, M, K, dev))
    return e


# ------------------------------------------------------------------ score

@pytest.mark.parametrize("dtype,B,M,K,pad,seed", [
    ("f32", 1, 128, 512, 0, 0),
    ("bf16", 1, 128, 512, 0, 1),
    ("bf16", 3, 37, 300, 0, 2),
    ("bf16", 2, 1000, 129, 3, 3),      # rows not 16-byte aligned: element path
    ("f32", 2, 257, 77, 1, 4),
    ("bf16", 1, 1, 1, 0, 5),
    ("bf16", 1, 5000, 8, 0, 6),
    ("bf16", 4, 64, 2000, 8, 7),
    ("f32", 1, 3000, 1030, 2, 8),
    ("bf16", 2, 1000, 300, 4, 9),      # 16-byte rows, K % 8 != 0: partial column group
    ("bf16", 1, 70, 1030, 2, 10),      # a split shorter than one 64-row tile
])
def test_score(dtype, B, M, K, pad, seed):
    dev = require_gpu()
    stored = wl.random_case(seed, (B, M, K + pad), dtype, n_outlier=max(1, K // 50))
    Xd = to_device(stored, dtype, dev)[:, :, :K]
    e = _energies_gpu(Xd, B, M, K, dev).cpu().numpy().reshape(B, K)
    X = wl.decode(stored, dtype).astype(np.float64)[:, :, :K]
    for b in range(B):
        check_energies(e[b], ro.column_energies(X[b]), M)


def test_score_integer_ties_are_exact():
    dev = require_gpu()
    stored = wl.integer_case(11, (2, 513, 260), -3, 3, "bf16")
    e = _energies_gpu(to_device(stored, "bf16", dev), 2, 513, 260, dev).cpu().numpy()
    X = wl.decode(stored, "bf16").astype(np.float64)
    want = np.concatenate([ro.column_energies(X[b]) for b in range(2)])
    assert np.array_equal(e, want)


def test_score_nonfinite_inputs_propagate():
    dev = require_gpu()
    x = np.random.default_rng(3).standard_normal((300, 40)).astype(np.float32)
    x[5, 3] = np.nan
    x[7, 9] = np.inf
    x[8, 10] = -np.inf
    x[9, 11] = np.float32(3e38)              # square overflows fp32, not float64
    stored = wl.f32_to_bf16_bits(x)
    e = _energies_gpu(to_device(stored, "bf16", dev), 1, 300, 40, dev).cpu().numpy()
    want = ro.column_energies(wl.decode(stored, "bf16"))
    check_energies(e, want, 300)
    assert np.isnan(e[3]) and np.isposinf(e[9]) and np.isposinf(e[10]) and np.isfinite(e[11])


def test_score_is_deterministic():
    dev = require_gpu()
    stored = wl.random_case(12, (1, 8192, 1024), "bf16", n_outlier=10)
    Xd = to_device(stored, "bf16", dev)
    runs = [_energies_gpu(Xd, 1, 8192, 1024, dev).cpu().numpy() for _ in range(3)]
    assert all(np.array_equal(runs[0], r) for r in runs[1:])


def _ld8(n):
    return (n + 7) // 8 * 8


@pytest.mark.parametrize("B,M,K,seed", [
    (1, 128, 512, 0), (2, 1000, 296, 1), (1, 8192, 1024, 2), (3, 37, 8, 3), (1, 64, 136, 4),
    (2, 200, 2048, 5),
])
def test_score_kmajor(B, M, K, seed):
    """Energies bit-identical to rmm_score; Xt an exact transpose of X."""
    dev = require_gpu()
    stored = wl.random_case(60 + seed, (B, M, K), "bf16", n_outlier=max(1, K // 50))
    Xd = to_device(stored, "bf16", dev)
    e1 = _energies_gpu(Xd, B, M, K, dev)
    ldxt = _ld8(M)
    Xt_full = torch.full((B, K, ldxt), -1.0, dtype=torch.bfloat16, device=dev)
    Xt = Xt_full[:, :, :M]
    e2 = torch.empty(B * K, dtype=torch.float64, device=dev)
    rmm.rmm_score_kmajor(Xd, e2, Xt, _score_ws(B, M, K, dev))
    assert torch.equal(e1, e2)
    got = Xt_full.view(torch.int16).cpu().numpy().view(np.uint16)
    assert np.array_equal(got[:, :, :M], np.ascontiguousarray(stored.transpose(0, 2, 1)))
    assert np.all(got[:, :, M:] == 0xbf80)          # padding columns untouched
    e_ref = ro.column_energies(wl.decode(stored, "bf16")[0].astype(np.float64))
    check_energies(e2.cpu().numpy()[:K], e_ref, M)


@pytest.mark.parametrize("B,M,K,pad,seed", [(2, 1000, 300, 4, 0), (1, 333, 1030, 2, 1)])
def test_score_kmajor_ragged_k(B, M, K, pad, seed):
    """K not a multiple of 8 (rows padded to 16 bytes): the last column group
    is partial; only the K real rows of Xt are written."""
    dev = require_gpu()
    stored = wl.random_case(80 + seed, (B, M, K + pad), "bf16", n_outlier=max(1, K // 50))
    Xd = to_device(stored, "bf16", dev)[:, :, :K]
    e1 = _energies_gpu(Xd, B, M, K, dev)
    ldxt = _ld8(M)
    Xt_flat = torch.full((B * K + 1, ldxt), -1.0, dtype=torch.bfloat16, device=dev)  # + sentinel row
    Xt = Xt_flat[:B * K].view(B, K, ldxt)[:, :, :M]
    e2 = torch.empty(B * K, dtype=torch.float64, device=dev)
    rmm.rmm_score_kmajor(Xd, e2, Xt, _score_ws(B, M, K, dev))
    assert torch.equal(e1, e2)
    flat = Xt_flat.view(torch.int16).cpu().numpy().view(np.uint16)
    got = flat[:B * K].reshape(B, K, ldxt)
    assert np.array_equal(got[:, :, :M], np.ascontiguousarray(stored[:, :, :K].transpose(0, 2, 1)))
    assert np.all(flat[B * K] == 0xbf80) and np.all(got[:, :, M:] == 0xbf80)
    for b in range(B):
        e_ref = ro.column_energies(wl.decode(stored[b, :, :K], "bf16").astype(np.float64))
        check_energies(e2.cpu().numpy()[b * K:(b + 1) * K], e_ref, M)


# ----------------------------------------------------------------- select

def _energy_case(seed, B, K):
    rng = np.random.default_rng(seed)
    e = rng.gamma(2.0, 1.0, size=(B, K))
    if K >= 8:
        # exact ties, zeros of both signs, infinities and NaNs
        e[:, rng.choice(K, size=K // 8, replace=False)] = e[0, 0]
        e[:, rng.choice(K, size=max(1, K // 16), replace=False)] = 0.0
        e[0, rng.choice(K, size=max(1, K // 32), replace=False)] = -0.0
        e[0, rng.integers(K)] = np.inf
        e[-1, rng.integers(K)] = np.nan
        e[-1, rng.integers(K)] = np.nan
    return e


@pytest.mark.parametrize("K", [1, 5, 64, 128, 256, 257, 1000, 2048, 3000, 4096, 8192,
                               10000, 16384, 20000, 28672, 32768, 40000])
def test_select_matches_oracle_bitwise(K):
    dev = require_gpu()
    B = 3
    e = _energy_case(K, B, K)
    ks = sorted({1, max(1, K // 3), K // 2 + 1, max(1, K - 1), K})
    ed = torch.from_numpy(e.ravel()).to(dev)
    for k in ks:
        idx = torch.empty(B * k, dtype=torch.int32, device=dev)
        rmm.rmm_select(ed, k, idx)
        got = idx.cpu().numpy().reshape(B, k)
        for b in range(B):
            assert np.array_equal(got[b], ro.topk_indices(e[b], k)), (K, k, b)


def test_select_all_equal_takes_lowest_indices():
    dev = require_gpu()
    for K in (7, 300, 5000):
        ed = torch.full((K,), 2.5, dtype=torch.float64, device=dev)
        for k in (1, K // 2, K):
            idx = torch.empty(k, dtype=torch.int32, device=dev)
            rmm.rmm_select(ed, k, idx)
            assert np.array_equal(idx.cpu().numpy(), np.arange(k))


def test_select_negative_and_extreme_values():
    dev = require_gpu()
    e = np.array([-1.0, -np.inf, 5e-324, np.finfo(np.float64).max, -0.0, 0.0, -2.0,
                  np.inf, -5e-324, 1.0])
    ed = torch.from_numpy(e).to(dev)
    for k in range(1, len(e) + 1):
        idx = torch.empty(k, dtype=torch.int32, device=dev)
        rmm.rmm_select(ed, k, idx)
        assert np.array_equal(idx.cpu().numpy(), ro.topk_indices(e, k)), k


# ------------------------------------------------------------ reduced GEMM

def _ascending(seed, B, K, k):
    rng = np.random.default_rng(seed)
    return np.stack([np.sort(rng.choice(K, size=k, replace=False)) for _ in range(B)])


@pytest.mark.parametrize("dtype,B,M,N,K,k,seed", [
    ("bf16", 1, 200, 72, 300, 37, 0),
    ("bf16", 2, 129, 100, 64, 64, 1),        # N*2 bytes not a 16-byte multiple
    ("bf16", 1, 256, 256, 1024, 1024, 2),    # identity list = dense product
    ("bf16", 1, 1, 8, 1, 1, 3),
    ("bf16", 1, 70, 1, 50, 13, 4),
    ("bf16", 3, 300, 520, 700, 333, 5),
    ("bf16", 1, 513, 257, 2048, 1, 6),
    ("f32", 1, 200, 72, 300, 37, 7),
    ("f32", 2, 65, 130, 100, 99, 8),
    ("f32", 1, 128, 512, 512, 256, 9),
])
def test_reduced_gemm(dtype, B, M, N, K, k, seed):
    dev = require_gpu()
    Xs = wl.random_case(seed, (B, M, K), dtype, n_outlier=max(1, K // 40))
    Ws = wl.random_case(seed + 100, (K, N), dtype, std=0.02)
    idx = _ascending(seed, B, K, k)
    Xd, Wd = to_device(Xs, dtype, dev), to_device(Ws, dtype, dev)
    Yd = torch.empty((B, M, N), dtype=torch_dtype(dtype), device=dev)
    rmm.rmm_reduced_gemm(Xd, Wd, torch.from_numpy(idx.astype(np.int32)).to(dev), Yd)
    Y = from_device(Yd)
    X, W = wl.decode(Xs, dtype).astype(np.float64), wl.decode(Ws, dtype).astype(np.float64)
    for b in range(B):
        ref = ro.reduced_matmul(X[b], W, idx[b])
        absprod = np.abs(X[b][:, idx[b]]) @ np.abs(W[idx[b], :])
        check_product(Y[b], ref, absprod, k, dtype)


@pytest.mark.parametrize("B,M,N,K,k,ldw_pad,seed", [
    (1, 2100, 4100, 3000, 1111, 0, 50),     # ragged M, N and k tails in 256x256 tiles
    (2, 2048, 2048, 4096, 2048, 0, 51),     # two selection units
    (1, 2048, 4098, 700, 300, 0, 52),       # W rows not 16-byte multiples
    (1, 4096, 2048, 1024, 1, 0, 53),        # k = 1
    (1, 2048, 4096, 1024, 1024, 8, 54),     # identity list, padded W rows
])
def test_reduced_gemm_large_tiles(B, M, N, K, k, ldw_pad, seed):
    dev = require_gpu()
    Xs = wl.random_case(seed, (B, M, K), "bf16", n_outlier=max(1, K // 100))
    Ws = wl.random_case(seed + 100, (K, N + ldw_pad), "bf16", std=0.02)
    idx = _ascending(seed, B, K, k)
    Xd = to_device(Xs, "bf16", dev)
    Wd = to_device(Ws, "bf16", dev)[:, :N]
    Yd = torch.empty((B, M, N), dtype=torch.bfloat16, device=dev)
    rmm.rmm_reduced_gemm(Xd, Wd, torch.from_numpy(idx.astype(np.int32)).to(dev), Yd)
    Y = from_device(Yd)
    X = wl.decode(Xs, "bf16").astype(np.float64)
    W = wl.decode(Ws, "bf16").astype(np.float64)[:, :N]
    for b in range(B):
        ref = ro.reduced_matmul(X[b], W, idx[b])
        absprod = np.abs(X[b][:, idx[b]]) @ np.abs(W[idx[b], :])
        check_product(Y[b], ref, absprod, k, "bf16")


@pytest.mark.parametrize("B,M,N,K,k,seed", [
    (1, 200, 72, 300, 37, 0),        # 128-wide tiles, ragged everything
    (2, 129, 104, 64, 64, 1),
    (1, 1, 8, 1, 1, 3),
    (3, 300, 520, 700, 333, 5),
    (1, 513, 264, 2048, 1, 6),
    (1, 2100, 4104, 3000, 1111, 50),  # 256-wide tiles, ragged M/N/k tails
    (2, 2048, 2048, 4096, 2048, 51),
    (1, 4096, 2048, 1024, 1, 53),
    (1, 2048, 4096, 1024, 1024, 54),
    (4, 8000, 128, 3000, 1111, 60),   # 256 x 128 tiles (N <= 128), ragged M and k
    (5, 6500, 72, 500, 333, 61),      # 256 x 128 tiles, N and M ragged
])
def test_reduced_gemm_kmajor(B, M, N, K, k, seed):
    """Oracle parity, and bit-identity with the row-major gather (same k order)."""
    dev = require_gpu()
    Xs = wl.random_case(seed, (B, M, K), "bf16", n_outlier=max(1, K // 40))
    Ws = wl.random_case(seed + 100, (K, N), "bf16", std=0.02)
    idx = _ascending(seed, B, K, k)
    ldxt = _ld8(M)
    Xt_host = np.zeros((B, K, ldxt), dtype=np.uint16)
    Xt_host[:, :, :M] = Xs.transpose(0, 2, 1)
    Xtd = to_device(Xt_host, "bf16", dev)[:, :, :M]
    Wd = to_device(Ws, "bf16", dev)
    idd = torch.from_numpy(idx.astype(np.int32)).to(dev)
    Y = torch.empty((B, M, N), dtype=torch.bfloat16, device=dev)
    rmm.rmm_reduced_gemm_kmajor(Xtd, Wd, idd, Y)
    Y_row = torch.empty_like(Y)
    rmm.rmm_reduced_gemm(to_device(Xs, "bf16", dev), Wd, idd, Y_row)
    assert torch.equal(Y.view(torch.int16), Y_row.view(torch.int16))
    Yn = from_device(Y)
    X, W = wl.decode(Xs, "bf16").astype(np.float64), wl.decode(Ws, "bf16").astype(np.float64)
    for b in range(B):
        ref = ro.reduced_matmul(X[b], W, idx[b])
        check_product(Yn[b], ref, np.abs(X[b][:, idx[b]]) @ np.abs(W[idx[b], :]), k, "bf16")


@pytest.mark.parametrize("pad", [3, 6, 10])
def test_reduced_gemm_kmajor_strided_y(pad):
    """256-wide tiles with Y rows longer than N, one per store path: an odd
    row stride (pad 3) stores element by element, a stride of 4 mod 8 (pad 6)
    in 8-byte pieces, a stride of 0 mod 8 (pad 10) stages whole-width tiles
    through LDS and stores 16-byte row pieces.  Nothing is written past
    column N."""
    dev = require_gpu()
    B, M, N, K, k = 3, 2050, 1030, 300, 150
    Xs = wl.random_case(60 + pad, (B, M, K), "bf16", n_outlier=8)
    Ws = wl.random_case(61 + pad, (K, N + 2), "bf16", std=0.02)     # W rows 16-byte aligned
    idx = _ascending(62 + pad, B, K, k)
    ldxt = _ld8(M)
    Xt_host = np.zeros((B, K, ldxt), dtype=np.uint16)
    Xt_host[:, :, :M] = Xs.transpose(0, 2, 1)
    Xtd = to_device(Xt_host, "bf16", dev)[:, :, :M]
    Yfull = torch.full((B, M, N + pad), 7.0, dtype=torch.bfloat16, device=dev)
    rmm.rmm_reduced_gemm_kmajor(Xtd, to_device(Ws, "bf16", dev)[:, :N],
                                torch.from_numpy(idx.astype(np.int32)).to(dev), Yfull[:, :, :N])
    Y = from_device(Yfull)
    assert np.all(Y[:, :, N:] == 7.0)
    X, W = wl.decode(Xs, "bf16").astype(np.float64), wl.decode(Ws, "bf16").astype(np.float64)[:, :N]
    for b in range(B):
        ref = ro.reduced_matmul(X[b], W, idx[b])
        check_product(Y[b, :, :N], ref, np.abs(X[b][:, idx[b]]) @ np.abs(W[idx[b], :]), k, "bf16")


def test_reduced_gemm_strided_operands():
    """Leading dimensions larger than the logical widths."""
    dev = require_gpu()
    B, M, N, K, k = 2, 150, 96, 200, 77
    Xs = wl.random_case(20, (B, M, K + 24), "bf16", n_outlier=4)
    Ws = wl.random_case(21, (K, N + 40), "bf16", std=0.02)
    idx = _ascending(22, B, K, k)
    Xd = to_device(Xs, "bf16", dev)[:, :, :K]
    Wd = to_device(Ws, "bf16", dev)[:, :N]
    Yfull = torch.zeros((B, M, N + 8), dtype=torch.bfloat16, device=dev)
    Yd = Yfull[:, :, :N]
    rmm.rmm_reduced_gemm(Xd, Wd, torch.from_numpy(idx.astype(np.int32)).to(dev), Yd)
    Y = from_device(Yfull)
    assert np.all(Y[:, :, N:] == 0)          # nothing written past N
    X = wl.decode(Xs, "bf16").astype(np.float64)[:, :, :K]
    W = wl.decode(Ws, "bf16").astype(np.float64)[:, :N]
    for b in range(B):
        ref = ro.reduced_matmul(X[b], W, idx[b])
        check_product(Y[b, :, :N], ref, np.abs(X[b][:, idx[b]]) @ np.abs(W[idx[b]]), k, "bf16")


# -------------------------------------------------------------- reduced QK

@pytest.mark.parametrize("dtype,batch,H,Hkv,Lq,Lk,D,r,causal,seed", [
    ("bf16", 2, 4, 2, 100, 130, 128, 0.25, True, 0),
    ("bf16", 1, 8, 8, 64, 64, 64, 1.0, True, 1),
    ("bf16", 1, 2, 1, 130, 70, 80, 0.2, True, 2),      # Lq > Lk: rows fully masked
    ("bf16", 1, 4, 4, 200, 300, 128, 0.5, False, 3),
    ("bf16", 1, 2, 2, 257, 257, 128, 0.75, True, 4),
    ("bf16", 1, 2, 1, 33, 40, 128, 0.001, True, 5),    # k = 1
    # Lk % 8 == 0: the row-streaming kernel, each register layout it has
    ("bf16", 1, 4, 2, 200, 264, 128, 0.75, True, 8),   # k = 96: 2x2 wave strips
    ("bf16", 2, 2, 1, 136, 256, 128, 1.0, True, 9),    # k = 128, Lk > Lq
    ("bf16", 1, 4, 1, 130, 136, 128, 0.5, False, 10),  # k = 64: one key strip per wave
    ("bf16", 1, 2, 2, 300, 320, 64, 0.5, True, 11),
    ("bf16", 1, 2, 2, 256, 128, 128, 0.3, True, 12),   # Lq > Lk: leading rows fully masked
    ("bf16", 2, 8, 2, 520, 520, 128, 0.5, True, 13),   # 256-key tiles: two and a tail of 8
    ("bf16", 1, 4, 4, 1000, 1000, 128, 0.25, True, 14),  # k = 32, four 256-key tiles, ragged
    ("f32", 1, 4, 2, 100, 130, 128, 0.5, True, 6),
    ("f32", 1, 2, 2, 70, 70, 64, 1.0, False, 7),
])
def test_reduced_qk(dtype, batch, H, Hkv, Lq, Lk, D, r, causal, seed):
    dev = require_gpu()
    Qf = wl.heavy_tailed_heads((seed, 300), batch * H, Lq, D)
    Kf = wl.heavy_tailed_heads((seed, 301), batch * Hkv, Lk, D)
    Qs, Ks = wl.encode(Qf, dtype), wl.encode(Kf, dtype)
    Q = wl.decode(Qs, dtype).astype(np.float64).reshape(batch, H, Lq, D)
    Kv = wl.decode(Ks, dtype).astype(np.float64).reshape(batch, Hkv, Lk, D)
    k = ro.retained_count(r, D)
    Qd = to_device(Qs, dtype, dev).reshape(batch, H, Lq, D)
    Kd = to_device(Ks, dtype, dev).reshape(batch, Hkv, Lk, D)
    # per-head selection on Q through the library
    e = _energies_gpu(Qd.reshape(batch * H, Lq, D), batch * H, Lq, D, dev)
    idx = torch.empty(batch * H * k, dtype=torch.int32, device=dev)
    rmm.rmm_select(e, k, idx)
    Sd = torch.empty((batch, H, Lq, Lk), dtype=torch_dtype(dtype), device=dev)
    rmm.rmm_reduced_qk(Qd, Kd, idx.reshape(batch, H, k), Sd, causal=causal)
    S = from_device(Sd)
    idx_np = idx.cpu().numpy().reshape(batch, H, k)
    e_np = e.cpu().numpy().reshape(batch * H, D)
    for b in range(batch):
        S_ref, idx_ref, e_ref = ro.rmm_qk(Q[b], Kv[b], r, causal)
        for h in range(H):
            check_energies(e_np[b * H + h], e_ref[h], Lq)
        check_index_sets(idx_np[b], idx_ref, e_ref, Lq)
        isclose_inf_pattern(S[b], S_ref)
        for h in range(H):
            g = ro.gqa_kv_head(h, H, Hkv)
            I = idx_ref[h]
            absprod = np.abs(Q[b, h][:, I]) @ np.abs(Kv[b, g][:, I]).T
            fin = np.isfinite(S_ref[h])
            check_product(S[b, h][fin], S_ref[h][fin], absprod[fin], k, dtype,
                          scale=1 / math.sqrt(D))


# ------------------------------------------------------------- rmm_linear

@pytest.mark.parametrize("r", [0.5, 1.0])
def test_linear_f32_single_layer(r):
    """128 tokens x 512 -> 512, fp32, 8 outlier channels x10 (seed 0)."""
    dev = require_gpu()
    wk = wl.WORKLOADS["linear_f32"]
    proj = wk.projections[0]
    Xs = wl.encode(wl.workload_input(wk, "x"), "f32")
    Ws = wl.encode(wl.workload_weight(wk, proj), "f32")
    Xd, Wd = to_device(Xs, "f32", dev), to_device(Ws, "f32", dev)
    k = rmm.rmm_retained_count(r, 512)
    Yd = torch.empty((128, 512), dtype=torch.float32, device=dev)
    idx = torch.empty(k, dtype=torch.int32, device=dev)
    rmm.rmm_linear(Xd, Wd, r, Yd, idx_out=idx)
    X, W = Xs.astype(np.float64), Ws.astype(np.float64)
    Y_ref, idx_ref, e_ref = ro.rmm(X, W, r)
    check_index_sets(idx.cpu().numpy()[None], idx_ref[None], e_ref[None], 128)
    check_product(from_device(Yd), Y_ref, np.abs(X[:, idx_ref]) @ np.abs(W[idx_ref]), k, "f32")


def test_linear_equals_separate_calls_bitwise():
    dev = require_gpu()
    B, M, N, K, r = 2, 333, 200, 640, 0.4
    Xd = to_device(wl.random_case(30, (B, M, K), "bf16", n_outlier=9), "bf16", dev)
    Wd = to_device(wl.random_case(31, (K, N), "bf16", std=0.02), "bf16", dev)
    k = rmm.rmm_retained_count(r, K)
    Y1 = torch.empty((B, M, N), dtype=torch.bfloat16, device=dev)
    i1 = torch.empty(B * k, dtype=torch.int32, device=dev)
    rmm.rmm_linear(Xd, Wd, r, Y1, idx_out=i1)
    e = _energies_gpu(Xd, B, M, K, dev)
    i2 = torch.empty(B * k, dtype=torch.int32, device=dev)
    rmm.rmm_select(e, k, i2)
    Y2 = torch.empty_like(Y1)
    rmm.rmm_reduced_gemm(Xd, Wd, i2.reshape(B, k), Y2)
    assert torch.equal(i1, i2)
    assert torch.equal(Y1.view(torch.int16), Y2.view(torch.int16))
    # the workspace-held index list path gives the same output
    Y3 = torch.empty_like(Y1)
    rmm.rmm_linear(Xd, Wd, r, Y3)
    assert torch.equal(Y1.view(torch.int16), Y3.view(torch.int16))
    # the K-major split calls (what rmm_linear runs for aligned bf16)
    Xt = torch.empty((B, K, _ld8(M)), dtype=torch.bfloat16, device=dev)[:, :, :M]
    e2 = torch.empty_like(e)
    rmm.rmm_score_kmajor(Xd, e2, Xt, _score_ws(B, M, K, dev))
    assert torch.equal(e, e2)
    Y4 = torch.empty_like(Y1)
    rmm.rmm_reduced_gemm_kmajor(Xt, Wd, i2.reshape(B, k), Y4)
    assert torch.equal(Y1.view(torch.int16), Y4.view(torch.int16))
    # rows that are not 16-byte multiples take the row-major path: same bits
    Xpad = torch.zeros((B, M, K + 3), dtype=torch.bfloat16, device=dev)
    Xpad[:, :, :K] = Xd
    Y5 = torch.empty_like(Y1)
    rmm.rmm_linear(Xpad[:, :, :K], Wd, r, Y5)
    assert torch.equal(Y1.view(torch.int16), Y5.view(torch.int16))


def test_linear_is_deterministic():
    dev = require_gpu()
    Xd = to_device(wl.random_case(40, (1, 2048, 2048), "bf16", n_outlier=20), "bf16", dev)
    Wd = to_device(wl.random_case(41, (2048, 1024), "bf16", std=0.02), "bf16", dev)
    outs = []
    for _ in range(3):
        Y = torch.empty((1, 2048, 1024), dtype=torch.bfloat16, device=dev)
        rmm.rmm_linear(Xd, Wd, 0.5, Y)
        outs.append(Y.view(torch.int16).clone())
    assert all(torch.equal(outs[0], o) for o in outs[1:])


def _first_break(lst, K):
    """1 + the first position of a list that is not strictly ascending within [0, K), else 0."""
    for t, v in enumerate(lst):
        if v < 0 or v >= K or (t > 0 and lst[t - 1] >= v):
            return t + 1
    return 0


@pytest.mark.parametrize("K,k", [(1000, 300), (40000, 12345), (7, 7), (1, 1)])
def test_check_indices(K, k):
    """rmm_check_indices on valid lists (sorted random subsets and the
    library's own TopK lists) and on lists with planted defects at the first,
    a middle and the last position."""
    dev = require_gpu()
    rng = np.random.default_rng(K + k)
    B = 8
    lists = np.stack([np.sort(rng.choice(K, k, replace=False)) for _ in range(B)]).astype(np.int32)
    if k > 1:
        lists[1, 0] = -1                         # below range at t = 0
        lists[2, k - 1] = K                      # past range at the end
        m = k // 2
        lists[3, m] = lists[3, m - 1]            # duplicate in the middle
        lists[4, m - 1], lists[4, m] = lists[4, m], lists[4, m - 1]   # descending pair
        lists[5, m] = K + 7                      # out of range, then a later defect too
        lists[5, k - 1] = lists[5, k - 2]
    else:
        lists[1, 0] = K
    want = np.array([_first_break(list(l), K) for l in lists], dtype=np.int32)
    bad = rmm.rmm_check_indices(torch.from_numpy(lists).to(dev), K)
    assert np.array_equal(bad.cpu().numpy(), want)
    assert want[0] == 0 and (k == 1 or np.all(want[1:6] > 0))
    # the library's own selections always pass
    e = torch.from_numpy(rng.standard_normal(B * K) ** 2).to(dev)
    sel = torch.empty(B * k, dtype=torch.int32, device=dev)
    rmm.rmm_select(e, k, sel)
    assert int(rmm.rmm_check_indices(sel.view(B, k), K).abs().sum()) == 0
