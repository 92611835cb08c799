"""Decode-step reduced product (rmm_reduced_gemv, M <= 8 rows per unit) on the
GPU against the oracle: ragged sizes, the single-slice and split paths, rows
that are not 16-byte aligned, batches of units with different index sets,
and the 8B layer's projections for one token per sequence.  All calls go
through the C-ABI."""
import numpy as np
import pytest
import torch

import paper_2608_13426_amd as rmm
import workloads as wl
from oracle import rmm_oracle as ro
from tests.gpu_util import check_index_sets, check_product, from_device, gpu, require_gpu, to_device

pytestmark = gpu


def _run(seed, B, M, N, K, r, pad=0, select_on_gpu=False):
    dev = require_gpu()
    Xs = wl.random_case(seed, (B, M, K), "bf16", n_outlier=max(1, K // 100))
    Ws = wl.random_case(seed + 1, (K, N + pad), "bf16", std=0.02)
    X = wl.decode(Xs, "bf16").astype(np.float64)
    W = wl.decode(Ws, "bf16").astype(np.float64)[:, :N]
    k = ro.retained_count(r, K)
    idx_ref = np.stack([ro.topk_indices(ro.column_energies(X[b]), k) for b in range(B)])
    Xd = to_device(Xs, "bf16", dev)
    Wd = to_device(Ws, "bf16", dev)[:, :N]
    if select_on_gpu:
        e = torch.empty(B * K, dtype=torch.float64, device=dev)
        ws = torch.empty(max(rmm.rmm_workspace_size(rmm.RMM_OP_SCORE, B, M, K), 1),
                         dtype=torch.uint8, device=dev)
        rmm.rmm_score(Xd, e, ws)
        idx = torch.empty(B * k, dtype=torch.int32, device=dev)
        rmm.rmm_select(e, k, idx)
        e_ref = np.stack([ro.column_energies(X[b]) for b in range(B)])
        assert check_index_sets(idx.cpu().numpy().reshape(B, k), idx_ref, e_ref, M,
                                exact_sums=(M == 1)) == 0
    else:
        idx = torch.from_numpy(idx_ref.astype(np.int32)).to(dev)
    Y = torch.full((B, M, N), 7.0, dtype=torch.bfloat16, device=dev)
    rmm.rmm_reduced_gemv(Xd, Wd, idx.view(B, k), Y)
    Yg = from_device(Y)
    for b in range(B):
        I = idx_ref[b]
        ref = ro.reduced_matmul(X[b], W, I)
        absprod = np.abs(X[b][:, I]) @ np.abs(W[I])
        check_product(Yg[b], ref, absprod, k, "bf16")
    return Xd, Wd, idx.view(B, k), Y


@pytest.mark.parametrize("B,M,N,K,r,pad,seed", [
    (1, 1, 4096, 4096, 0.5, 0, 0),       # one decode token, list split over slices
    (3, 2, 1000, 777, 0.25, 0, 1),       # ragged N and K
    (16, 1, 520, 300, 0.75, 0, 2),       # many units: one slice, Y written directly
    (2, 5, 2048, 1433, 0.5, 0, 3),       # 5 rows (8-row kernel)
    (1, 8, 33, 64, 1.0, 0, 4),           # N far below one 512-column chunk
    (1, 3, 700, 500, 0.5, 3, 5),         # rows of W not 16-byte aligned: element loads
    (4, 1, 1536, 2000, 0.001, 0, 6),     # k = 1
    (1, 4, 6144, 4096, 0.25, 0, 7),
])
def test_reduced_gemv(B, M, N, K, r, pad, seed):
    _run(seed, B, M, N, K, r, pad)


def test_reduced_gemv_after_gpu_selection():
    _run(8, 5, 1, 3000, 14336, 0.5, select_on_gpu=True)


def test_reduced_gemv_is_deterministic():
    Xd, Wd, idx, Y = _run(9, 2, 1, 4096, 4096, 0.5)
    Y2 = torch.empty_like(Y)
    rmm.rmm_reduced_gemv(Xd, Wd, idx, Y2)
    assert torch.equal(Y.view(torch.int16), Y2.view(torch.int16))


def test_reduced_gemv_matches_gemm_within_rounding():
    """The decode kernel and the general gathered GEMM compute the same
    product: they may differ only by fp32 summation order."""
    Xd, Wd, idx, Y = _run(10, 2, 3, 1000, 2000, 0.5)
    Y2 = torch.empty_like(Y)
    rmm.rmm_reduced_gemm(Xd, Wd, idx, Y2)
    a, b = Y.float(), Y2.float()
    assert torch.max(torch.abs(a - b)).item() <= 2.0 ** -7 * torch.max(torch.abs(b)).item()


@pytest.mark.parametrize("B", [1, 16])
def test_layer_8b_decode(B):
    """One decode step of the 8B layer's projections: B sequences, one token
    each (the first B tokens of the layer's activations as the current
    tokens), every projection group at r = 0.25, 0.5, 0.75 and 1."""
    dev = require_gpu()
    wk = wl.WORKLOADS["layer_8b"]
    groups = {}
    for p in wk.projections:
        groups.setdefault(p.input_name, []).append(p)
    for name, projs in groups.items():
        K = wk.inputs[name][0]
        bits = wl.f32_to_bf16_bits(wl.workload_input(wk, name, M=B))
        X = wl.decode(bits, "bf16").astype(np.float64)
        Wbits = np.concatenate([wl.f32_to_bf16_bits(wl.workload_weight(wk, p)) for p in projs], axis=1)
        W = wl.decode(Wbits, "bf16").astype(np.float64)
        N = W.shape[1]
        Xd = torch.from_numpy(bits.view(np.int16)).to(dev).view(torch.bfloat16).reshape(B, 1, K)
        Wd = torch.from_numpy(Wbits.view(np.int16)).to(dev).view(torch.bfloat16)
        e = torch.empty(B * K, dtype=torch.float64, device=dev)
        ws = torch.empty(max(rmm.rmm_workspace_size(rmm.RMM_OP_SCORE, B, 1, K), 1),
                         dtype=torch.uint8, device=dev)
        rmm.rmm_score(Xd, e, ws)
        Y = torch.empty((B, 1, N), dtype=torch.bfloat16, device=dev)
        e_ref = [ro.column_energies(X[b:b + 1]) for b in range(B)]
        for r in (0.25, 0.5, 0.75, 1.0):
            k = ro.retained_count(r, K)
            idx = torch.empty(B * k, dtype=torch.int32, device=dev)
            rmm.rmm_select(e, k, idx)
            idx_ref = np.stack([ro.topk_indices(e_ref[b], k) for b in range(B)])
            idx_np = idx.cpu().numpy().reshape(B, k)
            # a single token's energies are exact squares of bf16 values:
            # exact ties are common and resolve to the lower index on both
            # sides, so every set must match bit for bit
            check_index_sets(idx_np, idx_ref, np.stack(e_ref), 1, exact_sums=True)
            rmm.rmm_reduced_gemv(Xd, Wd, idx.view(B, k), Y)
            Yg = from_device(Y)
            for b in range(B):
                I = idx_ref[b]
                ref = ro.reduced_matmul(X[b:b + 1], W, I)
                absprod = np.abs(X[b:b + 1][:, I]) @ np.abs(W[I])
                check_product(Yg[b], ref, absprod, k, "bf16")
        del Xd, Wd, Y
    torch.cuda.empty_cache()


# ------------------------------------------------- selection for one token

def _tokens_case(seed, dtype, B, K, special=False, integers=False):
    if integers:
        stored = wl.integer_case(seed, (B, K), -3, 3, dtype)
    else:
        stored = wl.random_case(seed, (B, K), dtype, n_outlier=max(1, K // 100))
    if special:
        vals = wl.decode(stored, dtype).copy()
        rng = np.random.default_rng(seed)
        for b in range(B):
            pos = rng.choice(K, size=min(K, 6), replace=False)
            for p_, v in zip(pos, [np.nan, np.inf, -np.inf, -0.0, 0.0, np.nan]):
                vals[b, p_] = v
        stored = wl.encode(vals.astype(np.float32), dtype)
    return stored


@pytest.mark.parametrize("dtype,B,K,r,special,integers,seed", [
    ("bf16", 1, 4096, 0.5, False, False, 0),
    ("bf16", 16, 4096, 0.25, False, False, 1),
    ("bf16", 3, 14336, 0.75, False, False, 2),
    ("bf16", 1, 28672, 0.5, False, False, 3),
    ("bf16", 2, 40000, 0.5, False, False, 4),     # beyond the register path
    ("bf16", 4, 300, 0.5, False, True, 5),        # many exact ties
    ("bf16", 2, 1000, 0.3, True, False, 6),       # NaN, +-inf, +-0
    ("f32", 2, 4096, 0.5, False, False, 7),
    ("f32", 3, 777, 0.5, True, False, 8),
    ("bf16", 1, 1, 1.0, False, False, 9),
    ("bf16", 5, 64, 0.001, False, False, 10),     # k = 1
    ("bf16", 2, 32768, 0.5, False, True, 11),     # 32 keys per thread, many exact ties
    ("bf16", 2, 20000, 0.3, True, False, 12),     # 32 keys per thread, NaN, +-inf, +-0
])
def test_select_tokens(dtype, B, K, r, special, integers, seed):
    """Equals the oracle's TopK of x^2 and, bit for bit, rmm_score +
    rmm_select on the same single-row units."""
    dev = require_gpu()
    stored = _tokens_case(seed, dtype, B, K, special, integers)
    X = wl.decode(stored, dtype).astype(np.float64)
    k = ro.retained_count(r, K)
    Xd = to_device(stored, dtype, dev)
    idx = torch.empty(B * k, dtype=torch.int32, device=dev)
    rmm.rmm_select_tokens(Xd, k, idx)
    ref = np.stack([ro.topk_indices(ro.column_energies(X[b:b + 1]), k) for b in range(B)])
    assert np.array_equal(idx.cpu().numpy().reshape(B, k), ref)
    e = torch.empty(B * K, dtype=torch.float64, device=dev)
    ws = torch.empty(max(rmm.rmm_workspace_size(rmm.RMM_OP_SCORE, B, 1, K), 1),
                     dtype=torch.uint8, device=dev)
    rmm.rmm_score(Xd.reshape(B, 1, K), e, ws)
    idx2 = torch.empty_like(idx)
    rmm.rmm_select(e, k, idx2)
    assert torch.equal(idx, idx2)


def test_decode_step_graph_replay():
    """A decode step (token selection + reduced product for two projection
    inputs) captured as a HIP graph: every replay, with eager work and
    synchronisations in between, equals the eager step bit for bit."""
    dev = require_gpu()
    parts = []
    for seed, (K, N, r) in enumerate(((4096, 6144, 0.5), (14336, 4096, 0.25))):
        X = to_device(wl.random_case(40 + seed, (1, 1, K), "bf16", n_outlier=40), "bf16", dev)
        W = to_device(wl.random_case(50 + seed, (K, N), "bf16", std=0.02), "bf16", dev)
        k = ro.retained_count(r, K)
        ws = torch.empty(max(rmm.rmm_gemv_workspace_size(1, 1, N, k), 1), dtype=torch.uint8,
                         device=dev)
        parts.append((X, W, k, ws, torch.empty(k, dtype=torch.int32, device=dev),
                      torch.empty((1, 1, N), dtype=torch.bfloat16, device=dev)))

    def step():
        for X, W, k, ws, idx, Y in parts:
            rmm.rmm_select_tokens(X, k, idx)
            rmm.rmm_reduced_gemv(X, W, idx.view(1, k), Y, workspace=ws)

    step()
    torch.cuda.synchronize()
    eager = [(idx.clone(), Y.clone()) for *_, idx, Y in parts]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    other = torch.empty(100, dtype=torch.int32, device=dev)
    for rep in range(4):
        for *_, idx, Y in parts:            # clobber the outputs between replays
            idx.fill_(-1)
            Y.fill_(0)
        rmm.rmm_select_tokens(parts[0][0], 100, other)   # eager work in between
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for (ie, ye), (*_, idx, Y) in zip(eager, parts):
            assert torch.equal(idx, ie), rep
            assert torch.equal(Y.view(torch.int16), ye.view(torch.int16)), rep


def _decode_case(dev, groups_np, B, r):
    """groups_np: [(X bits [B, K], W bits [K, N])].  rmm_decode_step against
    the separate calls (bit for bit) and the oracle."""
    groups, sep = [], []
    for Xb, Wb in groups_np:
        K, N = Wb.shape
        k = ro.retained_count(r, K)
        Xd = torch.from_numpy(Xb.view(np.int16)).to(dev).view(torch.bfloat16)
        Wd = torch.from_numpy(Wb.view(np.int16)).to(dev).view(torch.bfloat16)
        idx = torch.full((B * k,), -1, dtype=torch.int32, device=dev)
        Y = torch.full((B, N), 9.0, dtype=torch.bfloat16, device=dev)
        groups.append((Xd, Wd, k, idx, Y))
        i2 = torch.empty_like(idx)
        Y2 = torch.empty_like(Y)
        rmm.rmm_select_tokens(Xd, k, i2)
        rmm.rmm_reduced_gemv(Xd.view(B, 1, K), Wd, i2.view(B, k), Y2.view(B, 1, N))
        sep.append((i2, Y2))
    rmm.rmm_decode_step(groups)
    # the products alone over the step's sets, into fresh outputs
    prod = [(Xd, Wd, k, idx, torch.full_like(Y, 7.0)) for Xd, Wd, k, idx, Y in groups]
    rmm.rmm_decode_products(prod)
    for (Xd, Wd, k, idx, Y), (i2, Y2), (Xb, Wb), p in zip(groups, sep, groups_np, prod):
        assert torch.equal(idx, i2), "sets differ from rmm_select_tokens"
        assert torch.equal(Y.view(torch.int16), Y2.view(torch.int16)), "products differ from rmm_reduced_gemv"
        assert torch.equal(p[4].view(torch.int16), Y.view(torch.int16)), "rmm_decode_products differs"
        X = wl.decode(Xb, "bf16").astype(np.float64)
        W = wl.decode(Wb, "bf16").astype(np.float64)
        e_ref = X * X                                   # one row: the exact energies
        idx_ref = np.stack([ro.topk_indices(e_ref[b], k) for b in range(B)])
        check_index_sets(idx.cpu().numpy(), idx_ref, e_ref, 1, exact_sums=True)
        Yg = from_device(Y)
        for b in range(B):
            I = idx_ref[b]
            check_product(Yg[b][None], ro.reduced_matmul(X[b][None], W, I),
                          np.abs(X[b][None][:, I]) @ np.abs(W[I]), k, "bf16")


@pytest.mark.parametrize("B,r,seed", [(1, 0.5, 0), (3, 0.25, 1), (2, 1.0, 2), (5, 0.001, 3)])
def test_decode_step_groups(B, r, seed):
    """Ragged groups (K, N not multiples of the chunk; a single-slice group)."""
    dev = require_gpu()
    # one group wider than 16384 channels (two chunks of 16 keys per thread),
    # one wider than 32768 (a selection launch of its own)
    shapes = [(1000, 1536), (4096, 520), (264, 72), (2048, 3000), (20000, 136), (33000, 72)]
    groups = [(wl.random_case(seed + 10 * i, (B, K), "bf16", n_outlier=max(1, K // 100)),
               wl.random_case(seed + 10 * i + 1, (K, N), "bf16", std=0.02)) for i, (K, N) in enumerate(shapes)]
    _decode_case(dev, groups, B, r)


@pytest.mark.parametrize("name,B,ratios", [("layer_8b", 1, (0.25, 0.5, 0.75, 1.0)),
                                           ("layer_8b", 16, (0.25, 0.5, 0.75, 1.0)),
                                           ("layer_70b", 1, (0.5,))])
def test_layer_decode_step(name, B, ratios):
    """A layer's four projection groups (q|k|v, o, gate|up, down) as one
    grouped decode step, B sequences: the 8B layer at every ratio, the 70B
    layer (down: 28672 channels, one-pass token selection with 32 keys per
    thread) at r = 0.5."""
    dev = require_gpu()
    wk = wl.WORKLOADS[name]
    by = {}
    for p in wk.projections:
        by.setdefault(p.input_name, []).append(p)
    groups = []
    for name, projs in by.items():
        Xb = wl.f32_to_bf16_bits(wl.workload_input(wk, name, M=B))
        Wb = np.concatenate([wl.f32_to_bf16_bits(wl.workload_weight(wk, p)) for p in projs], axis=1)
        groups.append((Xb, Wb))
    print(f"{name}: decode step, B={B}, r in {ratios}", flush=True)
    for r in ratios:
        _decode_case(dev, groups, B, r)
