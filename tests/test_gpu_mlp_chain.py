"""The reduced gate|up projection with the SwiGLU epilogue feeding the reduced
down projection (rmm_reduced_gemm_swiglu_kmajor), on the GPU.

The activation H = silu(g) * u is checked against the oracle's float64
products and activation within a bound derived from the arithmetic (fp32
accumulation of the retained products, the bf16 roundings of g, u, silu(g)
and H, the fp32 evaluation of silu).  The down projection's selection is
decided on the bf16 H, so the oracle takes the GPU's H as that projection's
input: its energies must be the exact sums of squares (within float64
rounding), its index set the oracle's TopK of them, its product within the
product bound."""
import math

import numpy as np
import pytest
import torch

import paper_2608_13426_amd as rmm
import workloads as wl
from oracle import rmm_oracle as ro
from tests.gpu_util import (U16, U32, check_energies, check_index_sets, check_product,
                            from_device, require_gpu, to_device)

pytestmark = pytest.mark.gpu

SENTINEL = 7.0
LIP = 1.0999        # max |silu'(x)| (attained near x = 2.4)


def _h_bound(g_ref, u_ref, ag, au, k):
    """|H_gpu - H*| for H* = silu(g*) u* (float64 oracle).  ag, au: the sums
    of |x||w| over the retained products of g and u."""
    dg = (U16 + 2 * U32) * np.abs(g_ref) + (k + 2) * U32 * ag * (1 + U16)
    du = (U16 + 2 * U32) * np.abs(u_ref) + (k + 2) * U32 * au * (1 + U16)
    s_ref = ro.silu(g_ref)
    # fp32 silu of the rounded g: Lipschitz move, the fp32 evaluation (well
    # inside 2^-20 relative to |g|), then the bf16 rounding of silu
    ds = LIP * dg + 2.0 ** -20 * (np.abs(g_ref) + dg)
    es = ds + U16 * (np.abs(s_ref) + ds)
    sb = np.abs(s_ref) + es
    # the fp32 product of two bf16 values is exact; H is rounded to bf16 once
    return sb * du + np.abs(u_ref) * es + U16 * sb * (np.abs(u_ref) + du) + 1e-300


def _run_chain(dev, X, Xbits, Wg, Wu, Wgbits, Wubits, r, pad, rows=None, down=None):
    """Score + TopK of X, the fused gate|up GEMM with the SwiGLU epilogue, then
    (optionally) TopK of H's energies and the down GEMM.  X [B, M, K]."""
    B, M, K = X.shape
    F = Wg.shape[1]
    Xd = to_device(Xbits, "bf16", dev).reshape(B, M, K)
    Xt = torch.empty((B, K, M), dtype=torch.bfloat16, device=dev)
    e = torch.empty(B * K, dtype=torch.float64, device=dev)
    ws = torch.empty(max(rmm.rmm_workspace_size(rmm.RMM_OP_SCORE, B, M, K), 1),
                     dtype=torch.uint8, device=dev)
    rmm.rmm_score_kmajor(Xd, e, Xt, ws)
    k = rmm.rmm_retained_count(r, K)
    idx = torch.empty(B * k, dtype=torch.int32, device=dev)
    rmm.rmm_select(e, k, idx)
    idx_ref = np.stack([ro.topk_indices(ro.column_energies(X[b]), k) for b in range(B)])
    e_ref = [ro.column_energies(X[b]) for b in range(B)]
    assert check_index_sets(idx.cpu().numpy().reshape(B, k), idx_ref, np.stack(e_ref), M) == 0
    Wgu = rmm.swiglu_weight_layout(to_device(Wgbits, "bf16", dev), to_device(Wubits, "bf16", dev))
    Hfull = torch.full((B, F, M + pad), SENTINEL, dtype=torch.bfloat16, device=dev)
    Ht = Hfull[:, :, :M]
    eh = torch.full((B, F), -1.0, dtype=torch.float64, device=dev)
    rmm.rmm_reduced_gemm_swiglu_kmajor(Xt, Wgu, idx.view(B, k), Ht, eh)
    if pad:
        assert bool((Hfull[:, :, M:] == SENTINEL).all()), "padding columns written"
    rows = np.arange(M) if rows is None else rows
    H, EH = [], []
    eh_np = eh.cpu().numpy()
    for b in range(B):
        Hg = from_device(Ht[b]).T                     # [M, F]: the down projection's input
        # the activation against the oracle on the chosen rows
        I = idx_ref[b]
        Xr = X[b][rows]
        g_ref = ro.reduced_matmul(Xr, Wg, I)
        u_ref = ro.reduced_matmul(Xr, Wu, I)
        h_ref = ro.swiglu(g_ref, u_ref)
        ag = np.abs(Xr[:, I]) @ np.abs(Wg[I])
        au = np.abs(Xr[:, I]) @ np.abs(Wu[I])
        err = np.abs(Hg[rows] - h_ref)
        bound = _h_bound(g_ref, u_ref, ag, au, k)
        bad = err > bound
        assert not bad.any(), f"{int(bad.sum())} activations outside the bound; worst excess " \
                              f"{float(np.max(err - bound)):.3e}"
        assert err.max() / max(np.abs(h_ref).max(), 1e-30) <= 2e-2
        # H's energies: exact sums of the squares of the GPU's bf16 H
        EH.append(ro.column_energies(Hg))
        check_energies(eh_np[b], EH[b], M)
        H.append(Hg)
    if down is not None:
        Wd, Wdbits, rd = down
        N = Wd.shape[1]
        kd = rmm.rmm_retained_count(rd, F)
        sel = torch.empty(B * kd, dtype=torch.int32, device=dev)
        rmm.rmm_select(eh.view(-1), kd, sel)
        Y = torch.empty((B, M, N), dtype=torch.bfloat16, device=dev)
        rmm.rmm_reduced_gemm_kmajor(Ht, to_device(Wdbits, "bf16", dev), sel.view(B, kd), Y)
        for b in range(B):
            eb = EH[b]
            sel_ref = ro.topk_indices(eb, kd)
            assert check_index_sets(sel.cpu().numpy().reshape(B, kd)[b][None], sel_ref[None],
                                    eb[None], M) == 0
            Hr = H[b][rows]
            Y_ref = ro.reduced_matmul(Hr, Wd, sel_ref)
            absprod = np.abs(Hr[:, sel_ref]) @ np.abs(Wd[sel_ref])
            check_product(from_device(Y[b][torch.from_numpy(rows).to(dev)]), Y_ref, absprod, kd, "bf16")
    return H


@pytest.mark.parametrize("B,M,K,F,r,pad,seed", [
    (1, 200, 296, 128, 0.5, 0, 0),      # one ragged row tile, K not a multiple of 16
    (1, 520, 256, 384, 1.0, 8, 1),      # three row tiles (the last of 8 rows), r = 1
    (2, 264, 320, 256, 0.25, 16, 2),    # two units
    (1, 64, 64, 128, 0.001, 0, 3),      # k = 1
])
def test_swiglu_chain(B, M, K, F, r, pad, seed):
    dev = require_gpu()
    print(f"case B={B} M={M} K={K} F={F} r={r} pad={pad}", flush=True)
    Xbits = wl.random_case(seed, (B * M, K), "bf16", n_outlier=max(1, K // 100))
    X = wl.decode(Xbits, "bf16").astype(np.float64).reshape(B, M, K)
    Wgbits = wl.random_case(seed + 10, (K, F), "bf16", std=0.1)
    Wubits = wl.random_case(seed + 20, (K, F), "bf16", std=0.1)
    Wdbits = wl.random_case(seed + 30, (F, 96), "bf16", std=0.05)
    Wg, Wu, Wd = (wl.decode(w, "bf16").astype(np.float64) for w in (Wgbits, Wubits, Wdbits))
    _run_chain(dev, X, Xbits, Wg, Wu, Wgbits, Wubits, r, pad, down=(Wd, Wdbits, 0.5))


def test_swiglu_matches_unfused_gemm():
    """The fused kernel's g and u are the plain GEMM's outputs bit for bit (same
    accumulation), so H equals the activation of the unfused chain's Y up to
    the fp32 evaluation of silu: here bf16(bf16(silu(g)) * u) is recomputed
    on the host from the plain GEMM's bf16 g and u with numpy float32 and
    must agree to two bf16 units in the last place everywhere (a silu value
    one unit apart on a rounding boundary moves the rounded product by at
    most two), and exactly almost everywhere."""
    dev = require_gpu()
    # 8 x 16 tiles of 256: the plain launch takes the same 256-tile kernel
    M, K, F, r = 2048, 512, 2048, 0.5
    Xbits = wl.random_case(40, (M, K), "bf16", n_outlier=5)
    Wgbits = wl.random_case(41, (K, F), "bf16", std=0.1)
    Wubits = wl.random_case(42, (K, F), "bf16", std=0.1)
    Xd = to_device(Xbits, "bf16", dev)
    Xt = torch.empty((K, M), dtype=torch.bfloat16, device=dev)
    e = torch.empty(K, dtype=torch.float64, device=dev)
    ws = torch.empty(max(rmm.rmm_workspace_size(rmm.RMM_OP_SCORE, 1, M, K), 1),
                     dtype=torch.uint8, device=dev)
    rmm.rmm_score_kmajor(Xd, e, Xt, ws)
    k = rmm.rmm_retained_count(r, K)
    idx = torch.empty(k, dtype=torch.int32, device=dev)
    rmm.rmm_select(e, k, idx)
    Wg, Wu = to_device(Wgbits, "bf16", dev), to_device(Wubits, "bf16", dev)
    Y = torch.empty((M, 2 * F), dtype=torch.bfloat16, device=dev)
    rmm.rmm_reduced_gemm_kmajor(Xt, torch.cat([Wg, Wu], dim=1).contiguous(), idx.view(1, k), Y)
    Ht = torch.empty((F, M), dtype=torch.bfloat16, device=dev)
    eh = torch.empty(F, dtype=torch.float64, device=dev)
    rmm.rmm_reduced_gemm_swiglu_kmajor(Xt, rmm.swiglu_weight_layout(Wg, Wu), idx.view(1, k), Ht, eh)
    g = Y[:, :F].float().cpu().numpy()
    u = Y[:, F:].float().cpu().numpy()
    s = torch.from_numpy((g / (np.float32(1) + np.exp(-g))).astype(np.float32)).bfloat16().float().numpy()
    want = torch.from_numpy((s * u).astype(np.float32)).bfloat16().float().numpy()
    got = Ht.float().cpu().numpy().T
    rel = np.abs(got - want) / (np.maximum(np.abs(want), np.abs(got)) + 1e-38)
    assert rel.max() <= 2.0 ** -6, f"worst relative difference {rel.max():.3e}"
    assert np.mean(got != want) < 0.01, f"{np.mean(got != want):.4f} of the values differ"


def test_swiglu_is_deterministic():
    dev = require_gpu()
    M, K, F = 264, 256, 128
    Xbits = wl.random_case(50, (M, K), "bf16")
    Xt = to_device(Xbits, "bf16", dev).t().contiguous()
    idx = torch.arange(0, K, 3, dtype=torch.int32, device=dev).view(1, -1)
    Wgu = to_device(wl.random_case(51, (K, 2 * F), "bf16", std=0.1), "bf16", dev)
    outs = []
    for _ in range(2):
        Ht = torch.empty((F, M), dtype=torch.bfloat16, device=dev)
        eh = torch.empty(F, dtype=torch.float64, device=dev)
        rmm.rmm_reduced_gemm_swiglu_kmajor(Xt, Wgu, idx, Ht, eh)
        outs.append((Ht, eh))
    assert torch.equal(outs[0][0].view(torch.int16), outs[1][0].view(torch.int16))
    assert torch.equal(outs[0][1], outs[1][1])


@pytest.mark.parametrize("name", ["layer_8b", "layer_70b"])
def test_layer_mlp_chain(name):
    """Full size, the launch configuration the benchmark times: the 8B MLP
    input [8192 x 4096] at r = 0.5 through gate|up [4096 x 14336 each] with
    the SwiGLU epilogue, then the down projection [14336 x 4096] at r = 0.5
    (the 70B layer: [16384 x 8192], 8192 -> 2 x 28672 -> 8192): index sets
    bit-exact, H's energies exact to float64 rounding, H and the down output
    on sampled rows against the oracle."""
    dev = require_gpu()
    wk = wl.WORKLOADS[name]
    print(f"{name}: gate|up with the SwiGLU epilogue -> down, r = 0.5", flush=True)
    Xbits = wl.f32_to_bf16_bits(wl.workload_input(wk, "mlp_in"))
    X = wl.decode(Xbits, "bf16").astype(np.float64)[None]
    proj = {p.name: p for p in wk.projections}
    Wgbits = wl.f32_to_bf16_bits(wl.workload_weight(wk, proj["gate"]))
    Wubits = wl.f32_to_bf16_bits(wl.workload_weight(wk, proj["up"]))
    Wdbits = wl.f32_to_bf16_bits(wl.workload_weight(wk, proj["down"]))
    Wg, Wu, Wd = (wl.decode(w, "bf16").astype(np.float64) for w in (Wgbits, Wubits, Wdbits))
    rng = np.random.default_rng(9)
    M = X.shape[1]
    rows = np.array(sorted({0, 1, 255, 256, M - 1} | set(int(v) for v in rng.choice(M, 19, replace=False))))
    _run_chain(dev, X, Xbits, Wg, Wu, Wgbits, Wubits, 0.5, 0, rows=rows, down=(Wd, Wdbits, 0.5))
    torch.cuda.empty_cache()


@pytest.mark.parametrize("r", [0.25, 0.5, 0.75, 1.0])
def test_mlp_1b_chain(r):
    """The 1B-class MLP shapes (2048 tokens, 2048 -> 2 x 8192 -> 2048) at every
    ratio of the sweep, with every row of H against the oracle."""
    dev = require_gpu()
    wk = wl.WORKLOADS["mlp_1b"]
    Xbits = wl.f32_to_bf16_bits(wl.workload_input(wk, "mlp_in"))
    X = wl.decode(Xbits, "bf16").astype(np.float64)[None]
    proj = {p.name: p for p in wk.projections}
    Wgbits = wl.f32_to_bf16_bits(wl.workload_weight(wk, proj["gate"]))
    Wubits = wl.f32_to_bf16_bits(wl.workload_weight(wk, proj["up"]))
    Wdbits = wl.f32_to_bf16_bits(wl.workload_weight(wk, proj["down"]))
    Wg, Wu, Wd = (wl.decode(w, "bf16").astype(np.float64) for w in (Wgbits, Wubits, Wdbits))
    _run_chain(dev, X, Xbits, Wg, Wu, Wgbits, Wubits, r, 0, down=(Wd, Wdbits, r))
