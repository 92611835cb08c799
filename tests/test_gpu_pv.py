"""Token-axis reduced value product (rmm_reduced_pv, Sec. 3.3) on the GPU
against the oracle: per query head the kt tokens with the largest column
norms of the attention weights P, then P[:, T] V[T, :] with the head's
shared value rows.  Index sets bit-exact (up to float64 near-ties, reported
by their margin), outputs within the product bound.  All calls go through
the C-ABI."""
import numpy as np
import pytest
import torch

import paper_2608_13426_amd as rmm
import workloads as wl
from oracle import rmm_oracle as ro
from tests.gpu_util import check_index_sets, check_product, from_device, gpu, require_gpu, to_device

pytestmark = gpu


def _weights(seed, H, Lq, Lk, causal):
    """Softmax rows of random scores (bottom-right causal mask), as float64."""
    S = wl.decode(wl.random_case(seed, (H, Lq, Lk), "f32"), "f32").astype(np.float64) * 2.0
    if causal:
        q = np.arange(Lq)[:, None]
        t = np.arange(Lk)[None, :]
        S = np.where(t > q + (Lk - Lq), -np.inf, S)
    S = S - S.max(axis=2, keepdims=True)
    E = np.where(np.isfinite(S), np.exp(S), 0.0)
    return E / E.sum(axis=2, keepdims=True)


def _run(seed, batch, H, Hkv, Lq, Lk, D, r, dtype, causal, pad=0):
    dev = require_gpu()
    Pv = np.stack([_weights(seed + b, H, Lq, Lk, causal) for b in range(batch)])
    Ps = wl.encode(np.pad(Pv, ((0, 0), (0, 0), (0, 0), (0, pad))).astype(np.float32), dtype)
    Vs = wl.random_case(seed + 50, (batch, Hkv, Lk, D), dtype)
    P = wl.decode(Ps, dtype).astype(np.float64)[..., :Lk]
    V = wl.decode(Vs, dtype).astype(np.float64)
    kt = ro.retained_count(r, Lk)
    Pd = to_device(Ps, dtype, dev)[..., :Lk]
    Vd = to_device(Vs, dtype, dev)
    O = torch.full((batch, H, Lq, D), 5.0, dtype=Vd.dtype, device=dev)
    idx = torch.empty(batch * H * kt, dtype=torch.int32, device=dev)
    rmm.rmm_reduced_pv(Pd, Vd, kt, O, idx_out=idx)
    Og = from_device(O)
    ig = idx.cpu().numpy().reshape(batch * H, kt)
    for b in range(batch):
        O_ref, idx_ref = ro.reduced_pv(P[b], V[b], kt)
        margins = [ro.selection_margin(ro.column_energies(P[b, h]), kt) for h in range(H)]
        check_index_sets(ig[b * H:(b + 1) * H], idx_ref, margins, Lq)
        for h in range(H):
            g = ro.gqa_kv_head(h, H, Hkv)
            T = idx_ref[h]
            absprod = np.abs(P[b, h][:, T]) @ np.abs(V[b, g][T])
            check_product(Og[b, h], O_ref[h], absprod, kt, dtype)
    return Pd, Vd, kt, O, idx


@pytest.mark.parametrize("batch,H,Hkv,Lq,Lk,D,r,dtype,causal,pad,seed", [
    (1, 4, 2, 100, 130, 64, 0.5, "bf16", False, 0, 0),     # ragged tokens, D = 64
    (2, 8, 2, 257, 257, 128, 0.25, "bf16", True, 0, 1),    # causal weights, 4 heads per kv head
    (1, 2, 1, 64, 300, 128, 1.0, "bf16", True, 0, 2),      # every token kept: the dense product
    (1, 4, 4, 70, 90, 32, 0.3, "f32", False, 0, 3),        # fp32
    (1, 2, 2, 33, 40, 128, 0.001, "bf16", True, 0, 4),     # kt = 1
    (1, 4, 2, 96, 200, 128, 0.5, "bf16", True, 5, 5),      # rows of P padded: row gather path
    (1, 8, 2, 512, 512, 128, 0.5, "bf16", True, 0, 6),     # 256-row tiles of the K-major path
])
def test_reduced_pv(batch, H, Hkv, Lq, Lk, D, r, dtype, causal, pad, seed):
    _run(seed, batch, H, Hkv, Lq, Lk, D, r, dtype, causal, pad)


def test_reduced_pv_is_deterministic_and_matches_steps():
    """Same result twice, and the same as the three entry points called in
    turn (rmm_score, rmm_select, rmm_reduced_gemm per kv head)."""
    dev = require_gpu()
    Pd, Vd, kt, O, idx = _run(7, 1, 4, 2, 128, 192, 128, 0.5, "bf16", True)
    O2 = torch.empty_like(O)
    idx2 = torch.empty_like(idx)
    rmm.rmm_reduced_pv(Pd, Vd, kt, O2, idx_out=idx2)
    assert torch.equal(idx, idx2) and torch.equal(O.view(torch.int16), O2.view(torch.int16))
    H, Lq, Lk = 4, 128, 192
    e = torch.empty(H * Lk, dtype=torch.float64, device=dev)
    ws = torch.empty(max(rmm.rmm_workspace_size(rmm.RMM_OP_SCORE, H, Lq, Lk), 1),
                     dtype=torch.uint8, device=dev)
    rmm.rmm_score(Pd.reshape(H, Lq, Lk), e, ws)
    idx3 = torch.empty_like(idx)
    rmm.rmm_select(e, kt, idx3)
    assert torch.equal(idx, idx3)
    O3 = torch.empty_like(O)
    for g in range(2):
        rmm.rmm_reduced_gemm(Pd[0, 2 * g:2 * g + 2].contiguous(), Vd[0, g],
                             idx3.view(H, kt)[2 * g:2 * g + 2].contiguous(), O3[0, 2 * g:2 * g + 2])
    a, b = O.float(), O3.float()
    assert torch.max(torch.abs(a - b)).item() <= 2.0 ** -7 * torch.max(torch.abs(b)).item()
