"""The reduced attention block writing the output projection's K-major input
and its column energies (rmm_reduced_attention_kmajor), on the GPU.

The block's values are those of rmm_reduced_attention (checked against the
oracle in test_gpu_attention.py); here the K-major copy must hold them bit for
bit, the energies must be the exact sums of their squares (within float64
rounding), and the chained output projection (TopK of those energies, then
the K-major gathered GEMM) must match the oracle.  The retained set of the
projection is decided by the bf16 outputs, so the oracle takes the same bf16
values (the GPU's) as that projection's input."""
import numpy as np
import pytest
import torch

import paper_2608_13426_amd as rmm
import workloads as wl
from oracle import rmm_oracle as ro
from tests.gpu_util import (NORM_TOL, attention_bound, check_energies, check_index_sets,
                            check_product, from_device, require_gpu, to_device)
from tests.test_gpu_attention import _case

pytestmark = pytest.mark.gpu

D = 128
SENTINEL = 7.0     # written into the padding columns of Ot, which must stay untouched


def _head_sets(Q, batch, H, k):
    return np.stack([np.stack([ro.topk_indices(ro.column_energies(Q[b, h]), k) for h in range(H)])
                     for b in range(batch)]).astype(np.int32)


def _both(dev, Qs, Ks, Vs, idx, batch, H, Hkv, Lq, Lk, causal, pad):
    """O from rmm_reduced_attention, and (Ot, energy) from the K-major entry point."""
    Qd = to_device(Qs, "bf16", dev).reshape(batch, H, Lq, D)
    Kd = to_device(Ks, "bf16", dev).reshape(batch, Hkv, Lk, D)
    Vd = to_device(Vs, "bf16", dev).reshape(batch, Hkv, Lk, D)
    idd = torch.from_numpy(idx).to(dev)
    O = torch.empty((batch, H, Lq, D), dtype=torch.bfloat16, device=dev)
    rmm.rmm_reduced_attention(Qd, Kd, Vd, idd, O, causal=causal)
    Ot = torch.full((batch, H * D, Lq + pad), SENTINEL, dtype=torch.bfloat16, device=dev)
    e = torch.full((batch, H * D), -1.0, dtype=torch.float64, device=dev)
    rmm.rmm_reduced_attention_kmajor(Qd, Kd, Vd, idd, Ot, e, causal=causal)
    return O, Ot, e


def _check_layout_and_energies(O, Ot, e, batch, H, Lq, pad):
    want = O.permute(0, 1, 3, 2).reshape(batch, H * D, Lq)
    assert torch.equal(Ot[:, :, :Lq].view(torch.int16), want.view(torch.int16)), "K-major copy differs"
    if pad:
        assert bool((Ot[:, :, Lq:] == SENTINEL).all()), "padding columns written"
    e_np = e.cpu().numpy()
    Xo = []
    for b in range(batch):
        # the projection's input: X_o[t][h*D + d] = O[b][h][t][d]
        X = from_device(O[b]).transpose(1, 0, 2).reshape(Lq, H * D)
        check_energies(e_np[b], ro.column_energies(X), Lq)
        Xo.append(X)
    return Xo


@pytest.mark.parametrize("batch,H,Hkv,Lq,Lk,r,causal,pad,seed", [
    (1, 4, 2, 200, 200, 0.5, True, 0, 0),
    (2, 2, 1, 136, 72, 0.25, True, 8, 1),      # Lq > Lk: leading rows of O are 0
    (1, 4, 4, 64, 300, 1.0, False, 0, 2),      # one query tile of 64 rows, key tail
    (1, 2, 1, 264, 320, 0.75, True, 16, 3),    # second query tile holds 8 rows
    (1, 8, 2, 704, 704, 0.5, True, 0, 4),      # 8 heads (heads grouped per XCD), 3 tiles
    (2, 8, 4, 304, 520, 0.25, True, 24, 5),    # Lk > Lq, 16 (batch, head) units
    (1, 2, 2, 8, 8, 0.001, False, 8, 6),       # k = 1, a single 8-query tile
])
def test_kmajor_output_and_energies(batch, H, Hkv, Lq, Lk, r, causal, pad, seed):
    dev = require_gpu()
    print(f"case b={batch} H={H}/{Hkv} Lq={Lq} Lk={Lk} r={r} causal={causal} pad={pad}", flush=True)
    Qs, Ks, Vs = _case(seed, batch, H, Hkv, Lq, Lk, D)
    Q = wl.decode(Qs, "bf16").astype(np.float64).reshape(batch, H, Lq, D)
    idx = _head_sets(Q, batch, H, ro.retained_count(r, D))
    O, Ot, e = _both(dev, Qs, Ks, Vs, idx, batch, H, Hkv, Lq, Lk, causal, pad)
    _check_layout_and_energies(O, Ot, e, batch, H, Lq, pad)


def _o_projection(dev, Ot, e, W, Lq, r):
    """TopK of the energies and the K-major gathered GEMM over the output
    projection's weight rows, as the chain runs it."""
    K = W.shape[0]
    k = rmm.rmm_retained_count(r, K)
    sel = torch.empty(k, dtype=torch.int32, device=dev)
    rmm.rmm_select(e.view(-1), k, sel)
    Y = torch.empty((Lq, W.shape[1]), dtype=torch.bfloat16, device=dev)
    rmm.rmm_reduced_gemm_kmajor(Ot[0][:, :Lq], W, sel.view(1, k), Y)
    return sel, Y, k


def test_chain_into_output_projection():
    """Block -> energies -> TopK -> reduced output projection, against the
    oracle: the block's outputs within the attention bound, the projection's
    set bit-exact and its product within the rounding bound."""
    dev = require_gpu()
    batch, H, Hkv, L, r, N = 1, 8, 2, 520, 0.5, 320
    Qs, Ks, Vs = _case(21, batch, H, Hkv, L, L, D)
    Q = wl.decode(Qs, "bf16").astype(np.float64).reshape(batch, H, L, D)
    K = wl.decode(Ks, "bf16").astype(np.float64).reshape(batch, Hkv, L, D)
    V = wl.decode(Vs, "bf16").astype(np.float64).reshape(batch, Hkv, L, D)
    idx = _head_sets(Q, batch, H, ro.retained_count(r, D))
    O, Ot, e = _both(dev, Qs, Ks, Vs, idx, batch, H, Hkv, L, L, True, 0)
    Xo = _check_layout_and_energies(O, Ot, e, batch, H, L, 0)[0]
    # the block against the oracle
    Og = from_device(O[0])
    ref = ro.reduced_attention(Q[0], K[0], V[0], idx[0], True)
    bound = attention_bound(Q[0], K[0], V[0], idx[0], True, D ** -0.5)
    err = np.abs(Og - ref)
    assert np.all(err <= bound[:, :, None] + 2.0 ** -8 * np.abs(ref)), float(err.max())
    assert err.max() / np.abs(ref).max() <= NORM_TOL["bf16"]
    # the output projection on the block's bf16 outputs
    Ws = wl.random_case(22, (H * D, N), "bf16", std=0.02)
    W = wl.decode(Ws, "bf16").astype(np.float64)
    sel, Y, k = _o_projection(dev, Ot, e, to_device(Ws, "bf16", dev), L, r)
    e_ref = ro.column_energies(Xo)
    sel_ref = ro.topk_indices(e_ref, k)
    assert check_index_sets(sel.cpu().numpy()[None], sel_ref[None], e_ref[None], L) == 0
    Y_ref = ro.reduced_matmul(Xo, W, sel_ref)
    absprod = np.abs(Xo[:, sel_ref]) @ np.abs(W[sel_ref])
    check_product(from_device(Y), Y_ref, absprod, k, "bf16")


def test_kmajor_is_deterministic():
    dev = require_gpu()
    Qs, Ks, Vs = _case(23, 1, 4, 2, 304, 304, D)
    idx = np.stack([np.arange(0, 128, 2, dtype=np.int32)] * 4)[None]
    _, Ot1, e1 = _both(dev, Qs, Ks, Vs, idx, 1, 4, 2, 304, 304, True, 8)
    _, Ot2, e2 = _both(dev, Qs, Ks, Vs, idx, 1, 4, 2, 304, 304, True, 8)
    assert torch.equal(Ot1.view(torch.int16), Ot2.view(torch.int16))
    assert torch.equal(e1, e2)


@pytest.mark.parametrize("name", ["layer_8b", "layer_70b"])
def test_layer_chain(name):
    """Full size, the launch configuration the benchmark times: the 8B
    attention shape (32 q / 8 kv heads, 8192 tokens, causal; the 70B layer:
    64 / 8 heads, 16384 tokens) at r = 0.5, then the output projection
    ([4096 x 4096]; [8192 x 8192]) at r = 0.5: K-major copy equal to the
    block's output, energies exact to float64 rounding, the projection's set
    bit-exact, its output on sampled rows against the oracle."""
    dev = require_gpu()
    wk = wl.WORKLOADS[name]
    print(f"{name}: attention block -> output projection, r = 0.5", flush=True)
    a = wk.attention
    q, kk = wl.workload_qk(wk)
    qb, kb = wl.f32_to_bf16_bits(q), wl.f32_to_bf16_bits(kk)
    vb = wl.f32_to_bf16_bits(wl.workload_v(wk))
    del q, kk
    Q = wl.decode(qb, "bf16").reshape(1, a.H, a.L, a.D)
    r = 0.5
    idx = _head_sets(Q, 1, a.H, ro.retained_count(r, a.D))
    O, Ot, e = _both(dev, qb, kb, vb, idx, 1, a.H, a.Hkv, a.L, a.L, True, 0)
    Xo = _check_layout_and_energies(O, Ot, e, 1, a.H, a.L, 0)[0]
    proj = next(p for p in wk.projections if p.name == "o")
    Wbits = wl.f32_to_bf16_bits(wl.workload_weight(wk, proj))
    W = wl.decode(Wbits, "bf16").astype(np.float64)
    sel, Y, k = _o_projection(dev, Ot, e, to_device(Wbits, "bf16", dev), a.L, r)
    e_ref = ro.column_energies(Xo)
    sel_ref = ro.topk_indices(e_ref, k)
    assert check_index_sets(sel.cpu().numpy()[None], sel_ref[None], e_ref[None], a.L) == 0
    rng = np.random.default_rng(8)
    rows = np.array(sorted({0, 1, 255, 256, a.L - 1} | set(int(v) for v in rng.choice(a.L, 27, replace=False))))
    Y_ref = ro.reduced_matmul(Xo[rows], W, sel_ref)
    absprod = np.abs(Xo[rows][:, sel_ref]) @ np.abs(W[sel_ref])
    check_product(from_device(Y[torch.from_numpy(rows).to(dev)]), Y_ref, absprod, k, "bf16")
    del O, Ot, e, Y
    torch.cuda.empty_cache()


def test_attn_4k_kmajor():
    """The 4k attention shape (32 heads, no GQA, heavy-tailed head dims,
    causal) at r = 0.5: the K-major copy equals the block's output, the
    energies are exact to float64 rounding."""
    dev = require_gpu()
    wk = wl.WORKLOADS["attn_4k"]
    a = wk.attention
    q, kk = wl.workload_qk(wk)
    qb, kb = wl.f32_to_bf16_bits(q), wl.f32_to_bf16_bits(kk)
    vb = wl.f32_to_bf16_bits(wl.workload_v(wk))
    del q, kk
    Q = wl.decode(qb, "bf16").reshape(1, a.H, a.L, a.D)
    idx = _head_sets(Q, 1, a.H, ro.retained_count(0.5, a.D))
    O, Ot, e = _both(dev, qb, kb, vb, idx, 1, a.H, a.Hkv, a.L, a.L, a.causal, 8)
    _check_layout_and_energies(O, Ot, e, 1, a.H, a.L, 8)
