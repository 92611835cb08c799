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
that read them would fail the product bound.

The same chain with the row statistics made by the scores' producer
(rmm_reduced_qk_rowstats -> rmm_attention_weights_kmajor_rowstats) runs on
integer-valued Q and K: every fp32 partial sum of their products is an
integer below 2^24, exact in any order, so the stored score is
bf16(fp32(acc * fp32(scale))) of the exact integer dot product acc, which
the oracle's float64 scores give back exactly.  The stored scores must then
match bit for bit, the row maxima exactly and the reciprocal sums within
the fp32 bound of their exponentials and sums, against the oracle's softmax
statistics of those scores."""
import math

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


def weights_bound(S_rows: np.ndarray, P_ref: np.ndarray, lanes=None) -> np.ndarray:
    """Per-element bound on |P_gpu - P*| for some query rows of one head
    (masked scores -inf).  With `lanes` the row statistics come from the
    scores' producer, whose sums are split over that many lanes per row and
    rescaled whenever their maximum rises: each rescaling's exponential errs
    by (2 shift + 4) u32 and the shifts along one partial sum add up to at
    most the row's spread."""
    out = np.zeros_like(P_ref)
    for n in range(S_rows.shape[0]):
        s = S_rows[n]
        keep = np.isfinite(s)
        if not keep.any():
            continue
        d = np.where(keep, s[keep].max() - np.where(keep, s, 0.0), 0.0)
        nk = int(keep.sum())
        rel = (2 * d + 4 + nk + 4) * U32
        if lanes is not None:
            rel = rel + (4 * d.max() + 4 * (nk / 8 + lanes + 8)) * U32
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


def _chain(dev, Sbits, Vbits, batch, H, Hkv, Lq, Lk, D, r, causal, pad=0, rows=None, heads=None,
           row_stats=None):
    """Run the chain and check every stage.  Sbits [batch, H, Lq, Lk] bf16
    bits of the scores (masked entries -inf when causal); row_stats: the
    (row_max, row_rinv) device tensors of those scores for the weights pass
    to use instead of its own, and the lanes per row that summed them."""
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
    if row_stats is None:
        rmm.rmm_attention_weights_kmajor(Sd, Pt, e, causal=causal)
    else:
        rmm.rmm_attention_weights_kmajor(Sd, Pt, e, causal=causal, row_max=row_stats[0],
                                         row_rinv=row_stats[1])
    lanes = None if row_stats is None else row_stats[2]
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
        bound = weights_bound(Srow, ref, lanes)
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


def exact_score_bits(Q: np.ndarray, K: np.ndarray, idx: np.ndarray, causal: bool,
                     rows=None) -> np.ndarray:
    """bf16 bits of the reduced scores of integer-valued Q [H, Lq, D] and K
    [Hkv, Lk, D] as stored with scale fp32(1/sqrt(D)): the oracle's float64
    scores times sqrt(D) give the integer dot products back exactly."""
    D = Q.shape[-1]
    acc = np.rint(ro.reduced_qk(Q, K, idx, causal, rows=rows) * math.sqrt(D))
    assert np.all(np.abs(acc[np.isfinite(acc)]) < 2.0 ** 24)
    return wl.f32_to_bf16_bits(acc.astype(np.float32) * np.float32(D ** -0.5))


def check_row_stats(rmax: np.ndarray, rinv: np.ndarray, S: np.ndarray, lanes: int):
    """GPU row statistics against the oracle's for the scores S [n, Lk]
    (float64, masked -inf).  The maximum is exact; the reciprocal sum errs
    by each exponential's (2|s - m| + 4) u32 (over every rescaling of a
    partial sum too: their shifts add up to at most the row's spread), the
    fp32 sums' n u32 and the reciprocal's u32; `lanes` threads share a
    row, each summing its 8-key chunks."""
    m_ref, r_ref = ro.softmax_row_stats(S)
    keep = np.isfinite(S)
    nk = keep.sum(axis=1)
    spread = np.where(nk > 0, m_ref - np.min(np.where(keep, S, np.inf), axis=1), 0.0)
    assert np.array_equal(rmax[nk == 0], np.zeros(int((nk == 0).sum())))
    assert np.array_equal(rinv[nk == 0], np.zeros(int((nk == 0).sum())))
    assert np.array_equal(rmax.astype(np.float64), m_ref), "row maximum differs"
    rel = (4 * spread + 4 * (nk / 8 + lanes + 8) + nk + 8) * U32
    err = np.abs(rinv.astype(np.float64) - r_ref)
    bad = err > rel * r_ref
    assert not bad.any(), f"{int(bad.sum())} reciprocal sums outside the bound; worst " \
                          f"{float(np.max(err / np.maximum(r_ref, 1e-300))):.3e} relative"


def _integer_qk(seed, batch, H, Hkv, Lq, Lk, D, k):
    Qb = wl.integer_case(seed, (batch, H, Lq, D), -3, 3, "bf16")
    Kb = wl.integer_case(seed + 1, (batch, Hkv, Lk, D), -3, 3, "bf16")
    rng = np.random.default_rng(seed)
    idx = np.stack([np.sort(rng.choice(D, k, replace=False)) for _ in range(batch * H)]).astype(np.int32)
    return Qb, Kb, idx


@pytest.mark.parametrize("batch,H,Hkv,Lq,Lk,D,k,causal,seed", [
    (1, 4, 2, 300, 304, 128, 64, True, 0),      # ragged query tile, Lk > Lq
    (1, 2, 1, 200, 264, 64, 32, True, 1),       # the D = 64 kernel
    (1, 2, 2, 320, 200, 128, 96, True, 2),      # Lq > Lk: leading rows keep nothing
    (2, 2, 1, 130, 392, 128, 128, False, 3),    # no mask, Lk not a multiple of the key tile
    (1, 2, 1, 1024, 1024, 128, 64, True, 4),    # several key tiles per row
    (1, 1, 1, 8, 8, 64, 1, True, 5),            # one partial tile, k = 1
])
def test_qk_rowstats_chain(batch, H, Hkv, Lq, Lk, D, k, causal, seed):
    dev = require_gpu()
    U = batch * H
    Qb, Kb, idx = _integer_qk(seed, batch, H, Hkv, Lq, Lk, D, k)
    Q = wl.decode(Qb, "bf16").reshape(batch, H, Lq, D)
    K = wl.decode(Kb, "bf16").reshape(batch, Hkv, Lk, D)
    ref = np.concatenate([exact_score_bits(Q[b], K[b], idx[b * H:(b + 1) * H], causal)
                          for b in range(batch)]).reshape(batch, H, Lq, Lk)
    Qd = to_device(Qb, "bf16", dev).reshape(batch, H, Lq, D)
    Kd = to_device(Kb, "bf16", dev).reshape(batch, Hkv, Lk, D)
    idx_d = torch.from_numpy(idx).to(dev).view(batch, H, k)
    S = torch.full((batch, H, Lq, Lk), float("nan"), dtype=torch.bfloat16, device=dev)
    rmax = torch.full((U * Lq,), float("nan"), dtype=torch.float32, device=dev)
    rinv = torch.full((U * Lq,), float("nan"), dtype=torch.float32, device=dev)
    rmm.rmm_reduced_qk_rowstats(Qd, Kd, idx_d, S, rmax, rinv, causal=causal)
    assert np.array_equal(S.view(torch.int16).cpu().numpy().view(np.uint16), ref), "stored scores differ"
    S2 = torch.empty_like(S)
    rmm.rmm_reduced_qk(Qd, Kd, idx_d, S2, causal=causal)
    assert torch.equal(S2.view(torch.int16), S.view(torch.int16))
    BT = 128 if (D == 64 or k > 96) else 256
    check_row_stats(rmax.cpu().numpy(), rinv.cpu().numpy(),
                    wl.decode(ref, "bf16").astype(np.float64).reshape(U * Lq, Lk), BT // 8)
    Vbits = wl.random_case(seed + 7, (batch, Hkv, Lk, D), "bf16")
    _chain(dev, ref, Vbits, batch, H, Hkv, Lq, Lk, D, 0.5, causal, row_stats=(rmax, rinv, BT // 8))


@pytest.mark.parametrize("r", [0.5, 1.0])
def test_layer_8b_qk_rowstats(r):
    """Full size, as the benchmark runs it: the 8B attention shape (32 query /
    8 kv heads, 8192 tokens, D = 128, causal) on integer-valued Q and K:
    stored scores of sampled query rows of every head bit for bit, every
    head's -inf count, the row statistics of those rows, and the weights the
    statistics give on those rows."""
    dev = require_gpu()
    a = wl.WORKLOADS["layer_8b"].attention
    k = ro.retained_count(r, a.D)
    print(f"Q [{a.H} x {a.L} x {a.D}], K [{a.Hkv} x {a.L} x {a.D}] integer, k = {k}", flush=True)
    Qb, Kb, idx = _integer_qk(80 + int(4 * r), 1, a.H, a.Hkv, a.L, a.L, a.D, k)
    Q = wl.decode(Qb, "bf16").reshape(a.H, a.L, a.D)
    K = wl.decode(Kb, "bf16").reshape(a.Hkv, a.L, a.D)
    rng = np.random.default_rng(205)
    rows = np.array(sorted({0, 1, 127, 128, 255, 256, a.L // 2, a.L - 2, a.L - 1} |
                           set(int(v) for v in rng.choice(a.L, 7, replace=False))))
    ref = exact_score_bits(Q, K, idx, True, rows=rows)                # [H, n, L]
    Qd = to_device(Qb, "bf16", dev).reshape(1, a.H, a.L, a.D)
    Kd = to_device(Kb, "bf16", dev).reshape(1, a.Hkv, a.L, a.D)
    S = torch.empty((1, a.H, a.L, a.L), dtype=torch.bfloat16, device=dev)
    rmax = torch.empty(a.H * a.L, dtype=torch.float32, device=dev)
    rinv = torch.empty(a.H * a.L, dtype=torch.float32, device=dev)
    rmm.rmm_reduced_qk_rowstats(Qd, Kd, torch.from_numpy(idx).to(dev).view(1, a.H, k), S, rmax, rinv,
                                causal=True)
    rows_d = torch.from_numpy(rows).to(dev)
    got = S[0][:, rows_d].view(torch.int16).cpu().numpy().view(np.uint16)
    assert np.array_equal(got, ref), "stored scores differ"
    n_inf = torch.isneginf(S[0]).sum(dim=(1, 2)).cpu().numpy()
    assert np.all(n_inf == a.L * (a.L - 1) // 2)
    sel = (np.arange(a.H)[:, None] * a.L + rows[None, :]).reshape(-1)
    Sref = wl.decode(ref, "bf16").astype(np.float64).reshape(-1, a.L)
    BT = 128 if k > 96 else 256
    check_row_stats(rmax.cpu().numpy()[sel], rinv.cpu().numpy()[sel], Sref, BT // 8)
    # the weights from these statistics on the sampled rows of every head
    Pt = torch.empty((1, a.H, a.L, a.L), dtype=torch.bfloat16, device=dev)
    e = torch.empty(a.H * a.L, dtype=torch.float64, device=dev)
    rmm.rmm_attention_weights_kmajor(S, Pt, e, causal=True, row_max=rmax, row_rinv=rinv)
    Pg = from_device(Pt[0][:, :, rows_d]).transpose(0, 2, 1)          # [H, n, L]
    Pg[:, unspecified(a.L, a.L, True)[rows]] = 0.0                    # zeros left unwritten
    Sref = Sref.reshape(a.H, rows.size, a.L)
    for h in range(a.H):
        P_ref = ro.attention_weights(Sref[h])
        err = np.abs(Pg[h] - P_ref)
        assert not (err > weights_bound(Sref[h], P_ref, BT // 8)).any(), f"head {h}"
    del S, Pt
    torch.cuda.empty_cache()
