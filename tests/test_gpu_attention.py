"""Reduced attention block on the GPU against the oracle (Sec. 3.3)."""
import math

import numpy as np
import pytest
import torch

import paper_2608_13426_amd as rmm
import workloads as wl
from oracle import rmm_oracle as ro
from tests.gpu_util import NORM_TOL, from_device, require_gpu, to_device

pytestmark = pytest.mark.gpu

U32 = 2.0 ** -24


def _case(seed, batch, H, Hkv, Lq, Lk, D):
    Qs = wl.encode(wl.heavy_tailed_heads((seed, 400), batch * H, Lq, D), "bf16")
    Ks = wl.encode(wl.heavy_tailed_heads((seed, 401), batch * Hkv, Lk, D), "bf16")
    Vs = wl.random_case(seed + 402, (batch * Hkv, Lk, D), "bf16")
    return Qs, Ks, Vs


def _bound(Q, K, V, idx, causal, D):
    """Per-row bound on |O - O_ref|: the weights are rounded to bf16 (2^-9) and
    shifted by the fp32 score error; the output is rounded to bf16."""
    H, Lq, _ = Q.shape
    Hkv, Lk, _ = K.shape
    k = idx.shape[1]
    out = np.empty((H, Lq))
    for h in range(H):
        g = ro.gqa_kv_head(h, H, Hkv)
        I = idx[h]
        mag = np.abs(Q[h][:, I]) @ np.abs(K[g][:, I]).T          # [Lq, Lk]
        err_s = (k + 4) * U32 * mag / math.sqrt(D)
        for i in range(Lq):
            keep = np.arange(Lk) <= (i + Lk - Lq) if causal else np.ones(Lk, bool)
            if not keep.any():
                out[h, i] = 0.0
                continue
            d = 2.0 ** -9 + 2.0 * err_s[i][keep].max()
            out[h, i] = 2.0 * d * np.abs(V[g][keep]).max()
    return out


@pytest.mark.parametrize("batch,H,Hkv,Lq,Lk,r,causal,seed", [
    (1, 4, 2, 200, 200, 0.5, True, 0),
    (2, 2, 1, 130, 70, 0.25, True, 1),        # Lq > Lk: leading rows fully masked -> 0
    (1, 4, 4, 64, 300, 1.0, False, 2),       # key tail past a 64-key tile
    (1, 2, 1, 257, 320, 0.75, True, 3),      # k = 96: two register k-groups
    (1, 8, 2, 128, 128, 0.001, True, 4),     # k = 1
    (1, 2, 2, 40, 40, 0.5, False, 5),
])
def test_reduced_attention(batch, H, Hkv, Lq, Lk, r, causal, seed):
    dev = require_gpu()
    D = 128
    Qs, Ks, Vs = _case(seed, batch, H, Hkv, Lq, Lk, D)
    Q = wl.decode(Qs, "bf16").astype(np.float64).reshape(batch, H, Lq, D)
    K = wl.decode(Ks, "bf16").astype(np.float64).reshape(batch, Hkv, Lk, D)
    V = wl.decode(Vs, "bf16").astype(np.float64).reshape(batch, Hkv, Lk, D)
    k = ro.retained_count(r, D)
    idx = np.stack([np.stack([ro.topk_indices(ro.column_energies(Q[b, h]), k) for h in range(H)])
                    for b in range(batch)]).astype(np.int32)
    Od = torch.full((batch, H, Lq, D), 3.0, dtype=torch.bfloat16, device=dev)
    rmm.rmm_reduced_attention(to_device(Qs, "bf16", dev).reshape(batch, H, Lq, D),
                              to_device(Ks, "bf16", dev).reshape(batch, Hkv, Lk, D),
                              to_device(Vs, "bf16", dev).reshape(batch, Hkv, Lk, D),
                              torch.from_numpy(idx).to(dev), Od, causal=causal)
    O = from_device(Od)
    for b in range(batch):
        ref = ro.reduced_attention(Q[b], K[b], V[b], idx[b], causal)
        bound = _bound(Q[b], K[b], V[b], idx[b], causal, D)
        err = np.abs(O[b] - ref)
        assert np.all(err <= bound[:, :, None] + 2.0 ** -8 * np.abs(ref)), float(err.max())
        denom = max(np.abs(ref).max(), 1e-30)
        assert err.max() / denom <= NORM_TOL["bf16"]
        if causal and Lq > Lk:
            assert np.all(O[b][:, :Lq - Lk] == 0.0)


def test_reduced_attention_matches_qk_softmax():
    """The fused block equals softmax of the library's own reduced QK^T times V
    (computed here in float64 from the bf16 scores): same scores, same mask."""
    dev = require_gpu()
    batch, H, Hkv, L, D, r = 1, 4, 2, 256, 128, 0.5
    Qs, Ks, Vs = _case(9, batch, H, Hkv, L, L, D)
    k = ro.retained_count(r, D)
    Q = wl.decode(Qs, "bf16").astype(np.float64).reshape(H, L, D)
    idx = np.stack([ro.topk_indices(ro.column_energies(Q[h]), k) for h in range(H)]).astype(np.int32)
    Qd = to_device(Qs, "bf16", dev).reshape(batch, H, L, D)
    Kd = to_device(Ks, "bf16", dev).reshape(batch, Hkv, L, D)
    Vd = to_device(Vs, "bf16", dev).reshape(batch, Hkv, L, D)
    idd = torch.from_numpy(idx).to(dev).reshape(batch, H, k)
    S = torch.empty((batch, H, L, L), dtype=torch.bfloat16, device=dev)
    rmm.rmm_reduced_qk(Qd, Kd, idd, S, causal=True)
    O = torch.empty((batch, H, L, D), dtype=torch.bfloat16, device=dev)
    rmm.rmm_reduced_attention(Qd, Kd, Vd, idd, O, causal=True)
    Sf = from_device(S)[0]
    V = wl.decode(Vs, "bf16").astype(np.float64).reshape(Hkv, L, D)
    Of = from_device(O)[0]
    for h in range(H):
        Vg = V[ro.gqa_kv_head(h, H, Hkv)]
        P = np.exp(Sf[h] - Sf[h].max(axis=1, keepdims=True))
        P /= P.sum(axis=1, keepdims=True)
        want = P @ Vg
        # the bf16 scores are within 2^-9 |S| of the fused kernel's fp32 ones, so
        # each weight moves by at most a factor exp(+-2 * 2^-9 max|S|) (plus the
        # fused kernel's own bf16 weights and output rounding)
        fin = np.where(np.isfinite(Sf[h]), np.abs(Sf[h]), 0.0).max(axis=1)
        d = 2.0 * 2.0 ** -9 * fin + 2.0 ** -8
        bound = 2.0 * np.expm1(d)[:, None] * np.abs(Vg).max() + 2.0 ** -8 * np.abs(want)
        assert np.all(np.abs(Of[h] - want) <= bound)


def test_reduced_attention_is_deterministic():
    dev = require_gpu()
    Qs, Ks, Vs = _case(11, 1, 4, 2, 300, 300, 128)
    idx = torch.stack([torch.arange(0, 128, 2, dtype=torch.int32)] * 4).to(dev).view(1, 4, 64)
    args = [to_device(Qs, "bf16", dev).reshape(1, 4, 300, 128),
            to_device(Ks, "bf16", dev).reshape(1, 2, 300, 128),
            to_device(Vs, "bf16", dev).reshape(1, 2, 300, 128), idx]
    O1 = torch.empty((1, 4, 300, 128), dtype=torch.bfloat16, device=dev)
    O2 = torch.empty_like(O1)
    rmm.rmm_reduced_attention(*args, O1)
    rmm.rmm_reduced_attention(*args, O2)
    assert torch.equal(O1.view(torch.int16), O2.view(torch.int16))
