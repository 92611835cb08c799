"""Reduced attention block on the GPU against the oracle (Sec. 3.3)."""
import math

import numpy as np
import pytest
import torch

import paper_2608_13426_amd as rmm
import workloads as wl
from oracle import rmm_oracle as ro
from tests.gpu_util import NORM_TOL, attention_bound, from_device, require_gpu, to_device

pytestmark = pytest.mark.gpu

U32 = 2.0 ** -24


def _case(seed, batch, H, Hkv, Lq, Lk, D):
    Qs = wl.encode(wl.heavy_tailed_heads((seed, 400), batch * H, Lq, D), "bf16")
    Ks = wl.encode(wl.heavy_tailed_heads((seed, 401), batch * Hkv, Lk, D), "bf16")
    Vs = wl.random_case(seed + 402, (batch * Hkv, Lk, D), "bf16")
    return Qs, Ks, Vs


def _run(seed, batch, H, Hkv, Lq, Lk, r, causal, scale=None):
    """GPU block against the oracle, element by element.  The oracle applies
    1/sqrt(D); another scale s is handed to it as Q * s * sqrt(D) (float64,
    an exact rewrite of the same scores)."""
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
                              torch.from_numpy(idx).to(dev), Od, causal=causal, scale=scale)
    O = from_device(Od)
    s = D ** -0.5 if scale is None else float(np.float32(scale))
    for b in range(batch):
        Qr = Q[b] * (s * math.sqrt(D))
        ref = ro.reduced_attention(Qr, K[b], V[b], idx[b], causal)
        bound = attention_bound(Q[b], K[b], V[b], idx[b], causal, s)
        err = np.abs(O[b] - ref)
        assert np.all(err <= bound[:, :, None] + 2.0 ** -8 * np.abs(ref)), float(err.max())
        denom = max(np.abs(ref).max(), 1e-30)
        assert err.max() / denom <= NORM_TOL["bf16"]
        if causal and Lq > Lk:
            assert np.all(O[b][:, :Lq - Lk] == 0.0)


@pytest.mark.parametrize("batch,H,Hkv,Lq,Lk,r,causal,seed", [
    (1, 4, 2, 200, 200, 0.5, True, 0),
    (2, 2, 1, 130, 70, 0.25, True, 1),        # Lq > Lk: leading rows fully masked -> 0
    (1, 4, 4, 64, 300, 1.0, False, 2),       # key tail past a 64-key tile
    (1, 2, 1, 257, 320, 0.75, True, 3),      # k = 96; two query tiles, the second of one row
    (1, 8, 2, 128, 128, 0.001, True, 4),     # k = 1
    (1, 2, 2, 40, 40, 0.5, False, 5),
    (1, 8, 2, 700, 700, 0.5, True, 6),       # 8 heads: heads grouped per XCD; three query tiles
    (2, 8, 4, 300, 520, 0.25, True, 7),      # Lk > Lq (bottom-right causal), 16 heads
    (1, 16, 2, 520, 520, 0.375, False, 8),   # k = 48, 16 heads, key tail
])
def test_reduced_attention(batch, H, Hkv, Lq, Lk, r, causal, seed):
    _run(seed, batch, H, Hkv, Lq, Lk, r, causal)


@pytest.mark.parametrize("scale", [-0.07, 0.0, 1.0, 3.0])
def test_reduced_attention_scales(scale):
    """Negative (Q negated), zero (uniform weights over the kept keys) and
    large scales (scores spanning many powers of two, so the running max is
    raised and O rescaled several times along a row)."""
    _run(12, 1, 4, 2, 300, 300, 0.5, True, scale=scale)


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
