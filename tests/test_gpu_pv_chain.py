"""The token-axis value product fed by its producer (Sec. 3.3): attention
scores -> rmm_attention_weights_kmajor (the softmax weights written K-major
with their token energies) -> rmm_select -> rmm_reduced_pv_kmajor, on the
GPU through the C-ABI.

The weights are checked element by element against the oracle's float64
softmax of the same bf16 scores within a bound derived from the arithmetic:
each exponential errs by (2|s - max| + 4) u32 relative (the fp32 argument,
the exp2 scaling and the hardware exp2), the fp32 row sum of n terms by
n u32, the reciprocal and the product by u32 each, then one bf16 rounding.
Masked weights are exactly 0.  The token selection is decided on those bf16
weights, so the oracle takes the GPU's weights as the value product's
input: the energies must be the exact sums of their squares (within float64
rounding), the token sets the oracle's TopK of them, the product within the
product bound.  With the causal flag the product skips the masked zeros;
the weights the producer leaves unwritten (zeros above the diagonal before
its 256-query block) are taken as zeros on the oracle's side, so a product
that read them would fail the product bound."""
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

SENTINEL = 3.0


def weights_bound(S_rows: np.ndarray, P_ref: np.ndarray) -> np.ndarray:
    """Per-element bound on |P_gpu - P*| for some query rows of one head
    (masked scores -inf)."""
    out = np.zeros_like(P_ref)
    for n in range(S_rows.shape[0]):
        s = S_rows[n]
        keep = np.isfinite(s)
        if not keep.any():
            continue
        d = np.where(keep, s[keep].max() - np.where(keep, s, 0.0), 0.0)
        nk = int(keep.sum())
        rel = (2 * d + 4 + nk + 4) * U32
        out[n] = ((1 + rel) * (1 + U16) - 1) * P_ref[n] + 1e-300
    return out


def unspecified(Lq: int, Lk: int, causal: bool) -> np.ndarray:
    """[Lq, Lk] True where the causal producer may leave Pt unwritten: masked
    (t > i + Lk - Lq) and before the 256-query block of column t's diagonal."""
    if not causal:
        return np.zeros((Lq, Lk), dtype=bool)
    i = np.arange(Lq)[:, None]
    d = np.arange(Lk)[None, :] - (Lk - Lq)
    return (i < d) & (i < 256 * np.floor_divide(d, 256))


def _chain(dev, Sbits, Vbits, batch, H, Hkv, Lq, Lk, D, r, causal, pad=0, rows=None, heads=None):
    """Run the chain and check every stage.  Sbits [batch, H, Lq, Lk] bf16
    bits of the scores (masked entries -inf when causal)."""
    U = batch * H
    Sb = Sbits.reshape(U, Lq, Lk)                       # decoded per checked head and row
    V = wl.decode(Vbits, "bf16").astype(np.float64).reshape(batch * Hkv, Lk, D)
    # score rows padded to a multiple of 8 elements; the padding holds NaN,
    # which must never be read
    lds = (Lk + 7) // 8 * 8
    Sfull = torch.full((batch, H, Lq, lds), float("nan"), dtype=torch.bfloat16, device=dev)
    Sfull[..., :Lk] = to_device(Sbits, "bf16", dev).reshape(batch, H, Lq, Lk)
    Sd = Sfull[..., :Lk]
    Vd = to_device(Vbits, "bf16", dev).reshape(batch, Hkv, Lk, D)
    ldpt = (Lq + 7) // 8 * 8 + pad
    full = torch.full((batch, H, Lk, ldpt), SENTINEL, dtype=torch.bfloat16, device=dev)
    Pt = full[..., :Lq]
    e = torch.full((U * Lk,), -1.0, dtype=torch.float64, device=dev)
    rmm.rmm_attention_weights_kmajor(Sd, Pt, e, causal=causal)
    if ldpt > Lq:
        assert bool((full[..., Lq:] == SENTINEL).all()), "padding columns written"
    rows = np.arange(Lq) if rows is None else np.asarray(rows)
    heads = range(U) if heads is None else heads
    Ptr = Pt.reshape(U, Lk, Lq)
    rows_d = torch.from_numpy(rows).to(dev)
    e_np = e.cpu().numpy().reshape(U, Lk)
    P_gpu = {}
    undef = unspecified(Lq, Lk, causal)
    for u in heads:
        Pu = from_device(Ptr[u]).T                        # [Lq, Lk]: the GPU's weights
        Pu[undef] = 0.0                                   # zeros by definition, left unwritten
        P_gpu[u] = Pu
        Srow = wl.decode(Sb[u][rows], "bf16").astype(np.float64)
        if causal:
            t = np.arange(Lk)[None, :]
            Srow = np.where(t > rows[:, None] + (Lk - Lq), -np.inf, Srow)
        ref = ro.attention_weights(Srow)
        err = np.abs(Pu[rows] - ref)
        bound = weights_bound(Srow, ref)
        bad = err > bound
        assert not bad.any(), f"head {u}: {int(bad.sum())} weights outside the bound; worst " \
                              f"excess {float(np.max(err - bound)):.3e}"
        assert np.array_equal(Pu[rows][ref == 0.0], np.zeros(int((ref == 0.0).sum()))), "masked weight not 0"
        check_energies(e_np[u], oracle_pool.column_energies(Pu), Lq)
    # token sets and the value product on the GPU's weights
    kt = ro.retained_count(r, Lk)
    idx = torch.empty(U * kt, dtype=torch.int32, device=dev)
    rmm.rmm_select(e, kt, idx)
    O = torch.full((batch, H, Lq, D), float("nan"), dtype=torch.bfloat16, device=dev)
    rmm.rmm_reduced_pv_kmajor(Pt, Vd, idx.view(U, kt), O, causal=causal)
    Og = from_device(O.reshape(U, Lq, D)[:, rows_d])
    ig = idx.cpu().numpy().reshape(U, kt)
    hl = list(heads)
    e_ref = np.stack([oracle_pool.column_energies(P_gpu[u]) for u in hl])
    T_ref = np.stack([ro.topk_indices(e_ref[n], kt) for n in range(len(hl))])
    assert check_index_sets(ig[hl], T_ref, e_ref, Lq) == 0
    for n, u in enumerate(hl):
        g = (u // H) * Hkv + (u % H) // (H // Hkv)
        T = T_ref[n]
        Pr = P_gpu[u][rows]
        ref = ro.reduced_matmul(Pr, V[g], T)
        check_product(Og[u], ref, np.abs(Pr[:, T]) @ np.abs(V[g][T]), kt, "bf16")
    return Pt, e, idx, O


@pytest.mark.parametrize("batch,H,Hkv,Lq,Lk,D,r,causal,pad,seed", [
    (1, 4, 2, 300, 300, 128, 0.5, True, 0, 0),      # ragged 64-query tiles, causal
    (2, 4, 1, 200, 264, 64, 0.25, True, 8, 1),      # Lk > Lq (bottom-right mask), padded Pt rows
    (1, 2, 2, 320, 200, 128, 0.75, True, 0, 2),     # Lq > Lk: leading rows fully masked
    (1, 4, 4, 130, 190, 128, 0.5, False, 0, 3),     # no mask
    (1, 2, 1, 96, 72, 32, 1.0, True, 0, 4),         # every token kept
    (1, 2, 1, 64, 64, 128, 0.001, True, 0, 5),      # kt = 1
    (1, 8, 2, 1024, 1024, 128, 0.5, True, 0, 6),    # 256-query tiles: the causal K-loop trimming
])
def test_pv_chain(batch, H, Hkv, Lq, Lk, D, r, causal, pad, seed):
    dev = require_gpu()
    Sbits = wl.attention_score_bits((seed, 500), batch * H, Lq, Lk, causal).reshape(batch, H, Lq, Lk)
    Vbits = wl.random_case(seed + 7, (batch, Hkv, Lk, D), "bf16")
    _chain(dev, Sbits, Vbits, batch, H, Hkv, Lq, Lk, D, r, causal, pad=pad)


def test_pv_chain_is_deterministic():
    dev = require_gpu()
    Sbits = wl.attention_score_bits((9, 500), 4, 512, 512, True).reshape(1, 4, 512, 512)
    Sd = to_device(Sbits, "bf16", dev).reshape(1, 4, 512, 512)
    res = []
    for fill in (0.0, 5.0):
        Pt = torch.full((1, 4, 512, 512), fill, dtype=torch.bfloat16, device=dev)
        e = torch.empty(4 * 512, dtype=torch.float64, device=dev)
        rmm.rmm_attention_weights_kmajor(Sd, Pt, e, causal=True)
        res.append((Pt, e))
    defined = torch.from_numpy(~unspecified(512, 512, True).T).to(dev)      # [t, i]
    assert torch.equal(res[0][0][0][:, defined].view(torch.int16), res[1][0][0][:, defined].view(torch.int16))
    assert torch.equal(res[0][1], res[1][1])


def test_layer_8b_pv_chain():
    """Full size, as the benchmark runs it: the 8B attention shape (32 query /
    8 kv heads, 8192 tokens, D = 128, causal) at rho_t = 0.5: weights of one
    head per kv head on sampled query rows, their energies, every head's
    token set and sampled output rows of those heads."""
    dev = require_gpu()
    wk = wl.WORKLOADS["layer_8b"]
    a = wk.attention
    print(f"scores [{a.H} x {a.L} x {a.L}] causal, V [{a.Hkv} x {a.L} x {a.D}]", flush=True)
    Sbits = wl.attention_score_bits((wk.seed, 204), a.H, a.L, a.L, True).reshape(1, a.H, a.L, a.L)
    Vbits = wl.f32_to_bf16_bits(wl.workload_v(wk)).reshape(1, a.Hkv, a.L, a.D)
    rng = np.random.default_rng(204)
    rows = np.array(sorted({0, 1, 255, 256, a.L // 2, a.L - 2, a.L - 1} |
                           set(int(v) for v in rng.choice(a.L, 9, replace=False))))
    heads = [4 * g + (g % 4) for g in range(a.Hkv)]
    _chain(dev, Sbits, Vbits, 1, a.H, a.Hkv, a.L, a.L, a.D, 0.5, True, rows=rows, heads=heads)
    torch.cuda.empty_cache()
