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
        e_ref = np.stack([ro.column_energies(P[b, h]) for h in range(H)])
        check_index_sets(ig[b * H:(b + 1) * H], idx_ref, e_ref, Lq)
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


def _sample_rows(L, n, seed):
    rng = np.random.default_rng(seed)
    fixed = {0, 1, 255, 256, L // 2, L - 2, L - 1}
    return np.array(sorted(fixed | set(int(v) for v in rng.choice(L, size=n, replace=False))))


def test_layer_8b_reduced_pv():
    """The 8B attention shape the benchmark times (32 query / 8 kv heads,
    8192 tokens, D = 128, causal attention weights): every head's token set
    bit-exact against the oracle, and every head's output on sampled query
    rows, at rho_t = 0.25, 0.5 and 1."""
    from tests import oracle_pool
    dev = require_gpu()
    wk = wl.WORKLOADS["layer_8b"]
    a = wk.attention
    H, Hkv, L, D = a.H, a.Hkv, a.L, a.D
    print(f"P [{H} x {L} x {L}] causal weights, V [{Hkv} x {L} x {D}]", flush=True)
    Pb = wl.attention_score_bits((wk.seed, 203), H, L, L, True, softmax=True)
    Vb = wl.f32_to_bf16_bits(wl.workload_v(wk))
    V = wl.decode(Vb, "bf16").astype(np.float64)
    Pd = torch.from_numpy(Pb.view(np.int16)).to(dev).view(torch.bfloat16).reshape(1, H, L, L)
    Vd = torch.from_numpy(Vb.view(np.int16)).to(dev).view(torch.bfloat16).reshape(1, Hkv, L, D)
    e_ref = np.stack([oracle_pool.column_energies(Pb[h], bf16_bits=True) for h in range(H)])
    rows = _sample_rows(L, 17, 203)
    rows_d = torch.from_numpy(rows).to(dev)
    Pr = wl.decode(Pb[:, rows], "bf16").astype(np.float64)          # [H, rows, L]
    O = torch.empty((1, H, L, D), dtype=torch.bfloat16, device=dev)
    ws = torch.empty(rmm.rmm_workspace_size(rmm.RMM_OP_PV, H, L, L, L), dtype=torch.uint8, device=dev)
    for r in (0.25, 0.5, 1.0):
        kt = ro.retained_count(r, L)
        idx = torch.empty(H * kt, dtype=torch.int32, device=dev)
        O.fill_(float("nan"))
        rmm.rmm_reduced_pv(Pd, Vd, kt, O, idx_out=idx, workspace=ws)
        idx_ref = np.stack([ro.topk_indices(e_ref[h], kt) for h in range(H)])
        assert check_index_sets(idx.cpu().numpy(), idx_ref, e_ref, L) == 0
        Og = from_device(O[0][:, rows_d])
        for h in range(H):
            g = ro.gqa_kv_head(h, H, Hkv)
            T = idx_ref[h]
            ref = ro.reduced_matmul(Pr[h], V[g], T)
            absprod = np.abs(Pr[h][:, T]) @ np.abs(V[g][T])
            check_product(Og[h], ref, absprod, kt, "bf16")
        print(f"rho_t={r}: kt={kt} ok", flush=True)
    del Pd, Vd, O, ws
    torch.cuda.empty_cache()
