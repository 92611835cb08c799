"""The RMSNorm producer of a reduced projection's input (rmm_rmsnorm_kmajor)
on the GPU, through the C-ABI.

Its K-major output is checked element by element against the oracle's
float64 RMSNorm within a bound derived from the arithmetic: the fp32 sum of
K exact squares, the division, eps and the reciprocal square root move the
row scale by at most (K/2 + 4) u32 relative, the fp32 product adds u32, and
the output is rounded to bf16 twice (the normalised value, then its product
with the weight).  The projection's selection is decided on those bf16
outputs, so the oracle takes the GPU's outputs as the projection's input:
their energies must be the exact sums of squares (within float64 rounding),
the index set the oracle's TopK of them, and the gathered product within
the product bound."""
import numpy as np
import pytest
import torch

import paper_2608_13426_amd as rmm
import workloads as wl
from oracle import rmm_oracle as ro
from tests import oracle_pool
from tests.gpu_util import (U16, U32, check_energies, check_index_sets, check_product,
                            from_device, require_gpu, to_device)

pytestmark = pytest.mark.gpu

SENTINEL = 7.0


def _gamma(seed, K):
    g = 1.0 + 0.3 * wl.normal_blocks((seed, 77), (1, K))[0]
    return wl.f32_to_bf16_bits(g)


def norm_bound(y_ref, K):
    d = (K / 2 + 4) * U32
    return ((1 + d) * (1 + U32) * (1 + U16) ** 2 - 1) * np.abs(y_ref) + 1e-300


def _run(dev, Xbits, gbits, eps, pad=0, rows=None, project=None):
    """X [B, M, K] bf16 bits -> the GPU's normalised rows [B, M, K] (float64)
    after checking them, their layout, energies and (optionally) the reduced
    projection that reads them: project = (W bits [K, N], r)."""
    B, M, K = Xbits.shape
    X = wl.decode(Xbits, "bf16").astype(np.float64)
    gamma = wl.decode(gbits, "bf16").astype(np.float64)
    Xd = to_device(Xbits, "bf16", dev)
    gd = to_device(gbits, "bf16", dev)
    ldxt = (M + 7) // 8 * 8 + pad            # Xt rows start 16-byte aligned
    full = torch.full((B, K, ldxt), SENTINEL, dtype=torch.bfloat16, device=dev)
    Xt = full[:, :, :M]
    e = torch.full((B * K,), -1.0, dtype=torch.float64, device=dev)
    rmm.rmm_rmsnorm_kmajor(Xd, gd, eps, Xt, e)
    if ldxt > M:
        assert bool((full[:, :, M:] == SENTINEL).all()), "padding columns written"
    rows = np.arange(M) if rows is None else np.asarray(rows)
    rows_d = torch.from_numpy(rows).to(dev)
    Y = []
    e_np = e.cpu().numpy().reshape(B, K)
    for b in range(B):
        Yb_rows = from_device(Xt[b][:, rows_d]).T                 # [rows, K]
        y_ref = ro.rmsnorm(X[b][rows], gamma, eps)
        err = np.abs(Yb_rows - y_ref)
        bad = err > norm_bound(y_ref, K)
        assert not bad.any(), f"{int(bad.sum())} outputs outside the bound; worst excess " \
                              f"{float(np.max(err - norm_bound(y_ref, K))):.3e}"
        Yb = from_device(Xt[b]).T                                  # [M, K], every row
        check_energies(e_np[b], oracle_pool.column_energies(Yb), M)
        Y.append(Yb)
    if project is not None:
        Wbits, r = project
        W = wl.decode(Wbits, "bf16").astype(np.float64)
        N = W.shape[1]
        k = rmm.rmm_retained_count(r, K)
        sel = torch.empty(B * k, dtype=torch.int32, device=dev)
        rmm.rmm_select(e, k, sel)
        Yd = torch.empty((B, M, N), dtype=torch.bfloat16, device=dev)
        rmm.rmm_reduced_gemm_kmajor(Xt, to_device(Wbits, "bf16", dev), sel.view(B, k), Yd)
        e_ref = np.stack([oracle_pool.column_energies(Y[b]) for b in range(B)])
        sel_ref = np.stack([ro.topk_indices(e_ref[b], k) for b in range(B)])
        # one row: each energy is one exact square, so ties are exact
        assert check_index_sets(sel.cpu().numpy(), sel_ref, e_ref, M, exact_sums=(M == 1)) == 0
        for b in range(B):
            Yr = Y[b][rows]
            ref = ro.reduced_matmul(Yr, W, sel_ref[b])
            absprod = np.abs(Yr[:, sel_ref[b]]) @ np.abs(W[sel_ref[b]])
            check_product(from_device(Yd[b][rows_d]), ref, absprod, k, "bf16")
    return Y, Xt, e


@pytest.mark.parametrize("B,M,K,eps,pad,seed", [
    (1, 300, 4096, 1e-5, 0, 0),      # ragged last 64-row tile
    (2, 70, 2048, 1e-6, 8, 1),       # two units, padded Xt rows
    (1, 33, 8192, 1e-5, 0, 2),       # fewer rows than one tile, 8192 channels
    (1, 1, 512, 0.0, 0, 3),          # one token, eps = 0
    (1, 130, 520, 10.0, 0, 4),       # K not a multiple of 64 (partial column strip); a large eps
    (4, 2000, 1024, 1e-5, 0, 5),     # four units, several row splits each
    (1, 9000, 256, 1e-5, 0, 6),      # many row splits of a narrow input
    (2, 512, 3072, 1e-5, 0, 7),      # 16 row blocks per unit (paired blocks), 3 column tiles per wave
])
def test_rmsnorm_kmajor(B, M, K, eps, pad, seed):
    dev = require_gpu()
    Xbits = wl.random_case(seed, (B, M, K), "bf16", n_outlier=max(1, K // 100), outlier_scale=20.0)
    _run(dev, Xbits, _gamma(seed, K), eps, pad=pad,
         project=(wl.random_case(seed + 9, (K, 192), "bf16", std=0.02), 0.5))


def test_rmsnorm_kmajor_equals_scoring_of_its_output():
    """The K-major output is the transpose of the normalised rows bit for
    bit: rmm_score_kmajor over the GPU's normalised rows (laid out row-major)
    writes the same Xt."""
    dev = require_gpu()
    B, M, K = 1, 264, 1024
    Xbits = wl.random_case(11, (B, M, K), "bf16", n_outlier=10, outlier_scale=20.0)
    Y, Xt, e = _run(dev, Xbits, _gamma(11, K), 1e-5)
    Yrow = Xt[0].t().contiguous()
    Xt2 = torch.empty_like(Xt[0])
    e2 = torch.empty(K, dtype=torch.float64, device=dev)
    ws = torch.empty(max(rmm.rmm_workspace_size(rmm.RMM_OP_SCORE, 1, M, K), 1), dtype=torch.uint8,
                     device=dev)
    rmm.rmm_score_kmajor(Yrow, e2, Xt2, ws)
    assert torch.equal(Xt2.view(torch.int16), Xt[0].view(torch.int16))
    check_energies(e.cpu().numpy(), ro.column_energies(Y[0]), M)
    check_energies(e2.cpu().numpy(), ro.column_energies(Y[0]), M)


def test_rmsnorm_kmajor_is_deterministic():
    dev = require_gpu()
    Xbits = wl.random_case(12, (1, 1000, 4096), "bf16", n_outlier=41, outlier_scale=20.0)
    gd = to_device(_gamma(12, 4096), "bf16", dev)
    Xd = to_device(Xbits, "bf16", dev)
    outs = []
    for _ in range(2):
        Xt = torch.empty((1, 4096, 1000), dtype=torch.bfloat16, device=dev)
        e = torch.empty(4096, dtype=torch.float64, device=dev)
        rmm.rmm_rmsnorm_kmajor(Xd, gd, 1e-5, Xt, e)
        outs.append((Xt, e))
    assert torch.equal(outs[0][0].view(torch.int16), outs[1][0].view(torch.int16))
    assert torch.equal(outs[0][1], outs[1][1])


@pytest.mark.parametrize("name", ["layer_8b", "layer_70b"])
def test_layer_rmsnorm_chain(name):
    """Full size, as the benchmark runs it: the attention input of the 8B
    (8192 x 4096) and 70B (16384 x 8192) layers through the norm producer,
    every energy and the q projection's set at r = 0.5, the normalised rows
    and the projection on sampled rows."""
    dev = require_gpu()
    wk = wl.WORKLOADS[name]
    K = wk.inputs["attn_in"][0]
    M = wk.M
    print(f"{name}: RMSNorm producer of the attention input, M={M} K={K}", flush=True)
    Xbits = wl.f32_to_bf16_bits(wl.workload_input(wk, "attn_in"))[None]
    proj = next(p for p in wk.projections if p.name == "q")
    Wbits = wl.f32_to_bf16_bits(wl.workload_weight(wk, proj))
    rng = np.random.default_rng(31)
    rows = np.array(sorted({0, 1, 255, 256, M // 2, M - 2, M - 1} |
                           set(int(v) for v in rng.choice(M, 24, replace=False))))
    _run(dev, Xbits, _gamma(31, K), 1e-5, rows=rows, project=(Wbits, 0.5))
    torch.cuda.empty_cache()
