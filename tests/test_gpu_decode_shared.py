"""Decode products over the union of a batch's sets
(rmm_decode_products_shared) on the GPU, through the C-ABI.

Every sequence's output is checked element by element against the oracle's
float64 reduced product over that sequence's own set, within the fp32
accumulation bound; the per-sequence kernel (rmm_decode_products) is checked
on the same sets the same way.  Cases: ragged groups (K not a multiple of the
512-index ranges, N not a multiple of the 128-column chunks, a single range
that writes Y directly), one to 32 sequences, identical, disjoint and
clustered sets (ranges with an empty union), one retained index, all of
them, the 8B layer's groups at full size, determinism and graph replay."""
import numpy as np
import pytest
import torch

import paper_2608_13426_amd as rmm
import workloads as wl
from oracle import rmm_oracle as ro
from tests.gpu_util import check_product, from_device, gpu, require_gpu

pytestmark = gpu


def _dev_bits(bits, dev):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(dev).view(torch.bfloat16)


def _topk_sets(Xb, k):
    X = wl.decode(Xb, "bf16").astype(np.float64)
    return np.stack([ro.topk_indices(X[b] * X[b], k) for b in range(X.shape[0])])


def _shared_case(dev, groups_np, sets, cols=None):
    """groups_np: [(X bits [B, K], W bits [K, N])], sets: [int array [B, k]]
    (ascending).  The shared-rows products and the per-sequence products
    against the oracle; cols: per group, the output columns checked
    (default all)."""
    groups, per = [], []
    for (Xb, Wb), I in zip(groups_np, sets):
        B, k = I.shape
        N = Wb.shape[1]
        Xd, Wd = _dev_bits(Xb, dev), _dev_bits(Wb, dev)
        idx = torch.from_numpy(I.astype(np.int32).reshape(-1)).to(dev)
        groups.append((Xd, Wd, k, idx, torch.full((B, N), 9.0, dtype=torch.bfloat16, device=dev)))
        per.append((Xd, Wd, k, idx, torch.full((B, N), 7.0, dtype=torch.bfloat16, device=dev)))
    rmm.rmm_decode_products_shared(groups)
    rmm.rmm_decode_products(per)
    for i, ((Xb, Wb), I, g, p) in enumerate(zip(groups_np, sets, groups, per)):
        X = wl.decode(Xb, "bf16").astype(np.float64)
        c = np.arange(Wb.shape[1]) if cols is None else cols[i]
        Wc = wl.decode(np.ascontiguousarray(Wb[:, c]), "bf16").astype(np.float64)
        Ys, Yp = from_device(g[4])[:, c], from_device(p[4])[:, c]
        for b in range(I.shape[0]):
            S = I[b]
            ref = ro.reduced_matmul(X[b][None], Wc, S)
            absprod = np.abs(X[b][None][:, S]) @ np.abs(Wc[S])
            check_product(Ys[b][None], ref, absprod, len(S), "bf16")
            check_product(Yp[b][None], ref, absprod, len(S), "bf16")
    return groups


@pytest.mark.parametrize("B,r,seed", [(1, 0.5, 0), (3, 0.25, 1), (16, 0.5, 2), (32, 0.25, 3),
                                      (5, 0.001, 4), (7, 1.0, 5)])
def test_shared_products_ragged_groups(B, r, seed):
    """Ragged groups: one range (K < 512), K just past a range, a ragged last
    range and column chunk, a wide group of 40 ranges, and eight channels
    with fewer columns than one chunk."""
    dev = require_gpu()
    shapes = [(296, 136), (520, 520), (2048, 3000), (1000, 1536), (20000, 200), (8, 24)]
    groups, sets = [], []
    for i, (K, N) in enumerate(shapes):
        Xb = wl.random_case(seed + 10 * i, (B, K), "bf16", n_outlier=max(1, K // 100))
        Wb = wl.random_case(seed + 10 * i + 1, (K, N), "bf16", std=0.02)
        groups.append((Xb, Wb))
        sets.append(_topk_sets(Xb, ro.retained_count(r, K)))
    _shared_case(dev, groups, sets)


def test_shared_products_set_structure():
    """Identical sets in every sequence, disjoint sets, sets packed into one
    range (the other ranges' unions are empty), the first and last index
    only, and a set covering every index."""
    dev = require_gpu()
    B, K, N = 8, 3000, 384
    rng = np.random.default_rng(61)
    Xb = wl.random_case(60, (B, K), "bf16", n_outlier=30)
    Wb = wl.random_case(62, (K, N), "bf16", std=0.02)
    same = np.tile(np.sort(rng.choice(K, 700, replace=False)), (B, 1))
    disjoint = np.stack([np.arange(b * 300, b * 300 + 300) for b in range(B)])
    packed = np.stack([np.sort(rng.choice(np.arange(1024, 1536), 200, replace=False)) for _ in range(B)])
    ends = np.tile(np.array([0, K - 1]), (B, 1))
    full = np.tile(np.arange(K), (B, 1))
    for I in (same, disjoint, packed, ends, full):
        _shared_case(dev, [(Xb, Wb)], [I])


@pytest.mark.parametrize("B,r,seed", [(4, 0.5, 90), (16, 0.25, 91), (32, 1.0, 92)])
def test_decode_step_shared(B, r, seed):
    """The batched step: its sets equal rmm_select_tokens' bit for bit, its
    outputs rmm_decode_products_shared's over those sets bit for bit (and so
    the oracle within the product bound); a group of more than 32768
    channels takes the generic selection."""
    dev = require_gpu()
    shapes = [(4096, 1024), (2048, 520), (33000, 72)]
    groups, ref = [], []
    for i, (K, N) in enumerate(shapes):
        Xb = wl.random_case(seed + 10 * i, (B, K), "bf16", n_outlier=max(1, K // 100))
        Wb = wl.random_case(seed + 10 * i + 1, (K, N), "bf16", std=0.02)
        Xd, Wd = _dev_bits(Xb, dev), _dev_bits(Wb, dev)
        k = ro.retained_count(r, K)
        idx = torch.full((B * k,), -1, dtype=torch.int32, device=dev)
        groups.append((Xd, Wd, k, idx, torch.full((B, N), 9.0, dtype=torch.bfloat16, device=dev)))
        i2 = torch.empty_like(idx)
        rmm.rmm_select_tokens(Xd.view(B, 1, K), k, i2)
        ref.append((Xd, Wd, k, i2, torch.full((B, N), 7.0, dtype=torch.bfloat16, device=dev)))
    rmm.rmm_decode_step_shared(groups)
    rmm.rmm_decode_products_shared(ref)
    for g, q in zip(groups, ref):
        assert torch.equal(g[3], q[3]), "sets differ from rmm_select_tokens"
        assert torch.equal(g[4].view(torch.int16), q[4].view(torch.int16)), "outputs differ"
    # the sets are the oracle's TopK of the exact squares; the products its
    # reduced products within the bound
    sets = [q[3].cpu().numpy().reshape(B, q[2]) for q in ref]
    groups_np = [(g[0].view(torch.int16).cpu().numpy().view(np.uint16),
                  g[1].view(torch.int16).cpu().numpy().view(np.uint16)) for g in groups]
    for (Xb, _), I in zip(groups_np, sets):
        assert np.array_equal(I, _topk_sets(Xb, I.shape[1]))
    _shared_case(dev, groups_np, sets)


def test_shared_products_deterministic_and_graph_replay():
    """Two calls give the same bits, and so does every replay of the call
    captured as a HIP graph (outputs clobbered, eager work in between)."""
    dev = require_gpu()
    B = 16
    shapes = [(4096, 1024), (14336, 512)]
    groups = []
    for i, (K, N) in enumerate(shapes):
        Xb = wl.random_case(70 + i, (B, K), "bf16", n_outlier=40)
        Wb = wl.random_case(80 + i, (K, N), "bf16", std=0.02)
        I = _topk_sets(Xb, ro.retained_count(0.5, K))
        groups.append((_dev_bits(Xb, dev), _dev_bits(Wb, dev), I.shape[1],
                       torch.from_numpy(I.astype(np.int32).reshape(-1)).to(dev),
                       torch.empty((B, N), dtype=torch.bfloat16, device=dev)))
    ws = torch.empty(rmm.rmm_decode_products_shared_workspace_size(groups), dtype=torch.uint8,
                     device=dev)
    rmm.rmm_decode_products_shared(groups, workspace=ws)
    first = [g[4].clone() for g in groups]
    rmm.rmm_decode_products_shared(groups, workspace=ws)
    for a, g in zip(first, groups):
        assert torch.equal(a.view(torch.int16), g[4].view(torch.int16))
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        rmm.rmm_decode_products_shared(groups, workspace=ws)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        rmm.rmm_decode_products_shared(groups, workspace=ws)
    other = torch.empty(64, dtype=torch.int32, device=dev)
    for rep in range(4):
        for g in groups:
            g[4].fill_(0)
        ws.fill_(255)                                 # stale workspace between replays
        rmm.rmm_select_tokens(groups[0][0][:1].reshape(1, 1, -1), 64, other)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for a, g in zip(first, groups):
            assert torch.equal(a.view(torch.int16), g[4].view(torch.int16)), rep


@pytest.mark.parametrize("name,B,r", [("layer_8b", 16, 0.5), ("layer_8b", 32, 0.25), ("layer_8b", 8, 1.0),
                                      ("layer_8b", 4, 0.5), ("layer_70b", 8, 0.5)])
def test_layer_shared_products(name, B, r):
    """A layer's four projection groups (q|k|v, o, gate|up, down) for B
    sequences at full size (8B: 4096 / 14336 channels; 70B: 8192 / 28672),
    each sequence's own TopK set; 512 sampled output columns of every group
    checked."""
    dev = require_gpu()
    wk = wl.WORKLOADS[name]
    by = {}
    for p in wk.projections:
        by.setdefault(p.input_name, []).append(p)
    groups, sets = [], []
    for name, projs in by.items():
        Xb = wl.f32_to_bf16_bits(wl.workload_input(wk, name, M=B))
        Wb = np.concatenate([wl.f32_to_bf16_bits(wl.workload_weight(wk, p)) for p in projs], axis=1)
        groups.append((Xb, Wb))
        sets.append(_topk_sets(Xb, ro.retained_count(r, Xb.shape[1])))
    print(f"{name} shared decode products B={B} r={r}", flush=True)
    rng = np.random.default_rng(5)
    cols = [np.unique(np.concatenate([[0, 127, 128, Wb.shape[1] - 1],
                                      rng.choice(Wb.shape[1], 508, replace=False)]))
            for _, Wb in groups]
    _shared_case(dev, groups, sets, cols=cols)
    torch.cuda.empty_cache()
