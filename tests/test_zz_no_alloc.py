"""rmm_linear_noalloc (the entry point for callers that cannot allocate
device memory) against rmm_linear on the same inputs, through the C-ABI:
index sets and outputs bit for bit, on calls in a row that reuse the one
scratch array of the GPU with shrinking sizes, plus the oracle on the last
call."""
import numpy as np
import pytest
import torch

import paper_2608_13426_amd as rmm
import workloads as wl
from oracle import rmm_oracle as ro
from tests.gpu_util import check_index_sets, check_product, from_device, gpu, require_gpu, to_device

pytestmark = gpu


def _pair(dev, seed, B, M, N, K, r, dtype, stream=None):
    Xs = wl.random_case(seed, (B, M, K), dtype, n_outlier=max(1, K // 100))
    Ws = wl.random_case(seed + 1, (K, N), dtype, std=0.02)
    Xd, Wd = to_device(Xs, dtype, dev), to_device(Ws, dtype, dev)
    k = rmm.rmm_retained_count(r, K)
    tdt = Xd.dtype
    Y1 = torch.full((B, M, N), 3.0, dtype=tdt, device=dev)
    Y2 = torch.full((B, M, N), -5.0, dtype=tdt, device=dev)
    i1 = torch.full((B * k,), -1, dtype=torch.int32, device=dev)
    i2 = torch.full((B * k,), -2, dtype=torch.int32, device=dev)
    rmm.rmm_linear(Xd, Wd, r, Y1, idx_out=i1, stream=stream)
    rmm.rmm_linear_noalloc(Xd, Wd, r, Y2, idx_out=i2, stream=stream)
    torch.cuda.synchronize()
    assert torch.equal(i1, i2), "index sets differ from rmm_linear"
    bits = torch.int16 if tdt == torch.bfloat16 else torch.int32
    assert torch.equal(Y1.view(bits), Y2.view(bits)), "outputs differ from rmm_linear"
    return Xs, Ws, i2, Y2, k


def test_noalloc_matches_linear_on_shrinking_calls():
    dev = require_gpu()
    cases = [  # (seed, B, M, N, K, r, dtype): each call smaller than the one before
        (0, 2, 1000, 1536, 2048, 0.5, "bf16"),
        (2, 1, 300, 520, 700, 0.25, "bf16"),
        (4, 1, 40, 72, 96, 0.75, "f32"),
    ]
    for seed, B, M, N, K, r, dtype in cases:
        print(f"rmm_linear_noalloc B={B} M={M} N={N} K={K} r={r} {dtype}", flush=True)
        Xs, Ws, idx, Y, k = _pair(dev, seed, B, M, N, K, r, dtype)
    # the last call against the oracle
    X = wl.decode(Xs, dtype).astype(np.float64)
    W = wl.decode(Ws, dtype).astype(np.float64)
    Yg = from_device(Y)
    e_ref = np.stack([ro.column_energies(X[b]) for b in range(B)])
    idx_ref = np.stack([ro.topk_indices(e_ref[b], k) for b in range(B)])
    assert check_index_sets(idx.cpu().numpy(), idx_ref, e_ref, M) == 0
    for b in range(B):
        I = idx_ref[b]
        check_product(Yg[b], ro.reduced_matmul(X[b], W, I), np.abs(X[b][:, I]) @ np.abs(W[I]), k, dtype)


def test_noalloc_on_a_side_stream():
    dev = require_gpu()
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        _pair(dev, 6, 1, 512, 640, 1024, 0.5, "bf16", stream=s)
        _pair(dev, 8, 2, 64, 256, 256, 1.0, "bf16", stream=s)


def test_noalloc_rejects_problems_beyond_its_scratch():
    dev = require_gpu()
    M, K, N = 8192, 4096, 64
    X = torch.zeros((M, K), dtype=torch.bfloat16, device=dev)
    W = torch.zeros((K, N), dtype=torch.bfloat16, device=dev)
    Y = torch.zeros((M, N), dtype=torch.bfloat16, device=dev)
    assert rmm.rmm_workspace_size(rmm.RMM_OP_LINEAR, 1, M, K, K // 2) > rmm.rmm_noalloc_scratch_bytes()
    with pytest.raises(rmm.RmmError) as ex:
        rmm.rmm_linear_noalloc(X, W, 0.5, Y)
    assert ex.value.status == 5
