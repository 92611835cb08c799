"""GPU parity at the workloads' full sizes, in the launch configuration the
benchmark times: every index set is compared with the oracle's (bit-exact
under the float64 margin rule), every energy within its rounding bound, and
outputs on sampled rows that the oracle computes one by one (including the
first and last rows, so tile tails are covered)."""
import functools
import zlib

import numpy as np
import pytest
import torch

import paper_2608_13426_amd as rmm
import workloads as wl
from oracle import rmm_oracle as ro
from tests import oracle_pool
from tests.gpu_util import (NORM_TOL, attention_bound, gpu, require_gpu, from_device,
                            check_energies, check_index_sets, check_product, isclose_inf_pattern)

pytestmark = gpu


def _rows(M, n, seed):
    rng = np.random.default_rng(seed)
    fixed = {0, 1, 255, 256, M // 2, M - 2, M - 1}
    rest = rng.choice(M, size=n, replace=False)
    return np.array(sorted(fixed | set(int(v) for v in rest)))


@functools.lru_cache(maxsize=4)
def _input(name, inp):
    """Stored bf16 bits and exact oracle energies of one activation input."""
    wk = wl.WORKLOADS[name]
    bits = wl.f32_to_bf16_bits(wl.workload_input(wk, inp))
    X = wl.decode(bits, "bf16")
    return bits, X, oracle_pool.column_energies(X)


def head_energies(Q: np.ndarray) -> np.ndarray:
    """The oracle's column energies of every head's Q [H x L x D] -> [H x D]:
    the columns of the [L x H*D] side-by-side layout are the heads' columns."""
    H, L, D = Q.shape
    return oracle_pool.column_energies(Q.transpose(1, 0, 2).reshape(L, H * D)).reshape(H, D)


def _dev_bf16(bits, dev):
    return torch.from_numpy(bits.view(np.int16)).to(dev).view(torch.bfloat16)


def _projection_case(name, proj_name, ratios):
    dev = require_gpu()
    wk = wl.WORKLOADS[name]
    proj = next(p for p in wk.projections if p.name == proj_name)
    bits, X, e_ref = _input(name, proj.input_name)
    M, K, N = wk.M, proj.K, proj.N
    Wbits = wl.f32_to_bf16_bits(wl.workload_weight(wk, proj))
    W = wl.decode(Wbits, "bf16")
    Xd, Wd = _dev_bf16(bits, dev), _dev_bf16(Wbits, dev)
    ws = torch.empty(max(rmm.rmm_workspace_size(rmm.RMM_OP_SCORE, 1, M, K), 1),
                     dtype=torch.uint8, device=dev)
    e = torch.empty(K, dtype=torch.float64, device=dev)
    rmm.rmm_score(Xd, e, ws)
    check_energies(e.cpu().numpy(), e_ref, M)
    rows = _rows(M, 57, zlib.crc32(f"{name}/{proj_name}".encode()))
    Y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
    for r in ratios:
        k = rmm.rmm_retained_count(r, K)
        idx = torch.empty(k, dtype=torch.int32, device=dev)
        rmm.rmm_select(e, k, idx)
        idx_ref = ro.topk_indices(e_ref, k)
        # no unit of these workloads sits within float64 rounding of a tie
        assert check_index_sets(idx.cpu().numpy()[None], idx_ref[None], e_ref[None], M) == 0
        rmm.rmm_reduced_gemm(Xd, Wd, idx.view(1, k), Y)
        Ys = from_device(Y[torch.from_numpy(rows).to(dev)])
        ref = ro.reduced_matmul(X[rows], W, idx_ref)
        absprod = np.abs(X[rows][:, idx_ref]).astype(np.float64) @ np.abs(W[idx_ref]).astype(np.float64)
        check_product(Ys, ref, absprod, k, "bf16")
        # the fused entry point gives the same bits
        Y2 = torch.empty_like(Y)
        i2 = torch.empty_like(idx)
        rmm.rmm_linear(Xd, Wd, r, Y2, idx_out=i2)
        assert torch.equal(i2, idx)
        assert torch.equal(Y2.view(torch.int16), Y.view(torch.int16))
    del Xd, Wd, Y
    torch.cuda.empty_cache()


def _attention_case(name, ratios, heads=None, n_rows=13):
    dev = require_gpu()
    wk = wl.WORKLOADS[name]
    a = wk.attention
    q, kk = wl.workload_qk(wk)
    qb, kb = wl.f32_to_bf16_bits(q), wl.f32_to_bf16_bits(kk)
    Q, Kc = wl.decode(qb, "bf16"), wl.decode(kb, "bf16")
    del q, kk
    Qd = _dev_bf16(qb, dev).reshape(1, a.H, a.L, a.D)
    Kd = _dev_bf16(kb, dev).reshape(1, a.Hkv, a.L, a.D)
    e_ref = head_energies(Q)
    ws = torch.empty(max(rmm.rmm_workspace_size(rmm.RMM_OP_SCORE, a.H, a.L, a.D), 1),
                     dtype=torch.uint8, device=dev)
    e = torch.empty(a.H * a.D, dtype=torch.float64, device=dev)
    rmm.rmm_score(Qd.reshape(a.H, a.L, a.D), e, ws)
    e_np = e.cpu().numpy().reshape(a.H, a.D)
    for h in range(a.H):
        check_energies(e_np[h], e_ref[h], a.L)
    S = torch.empty((1, a.H, a.L, a.L), dtype=torch.bfloat16, device=dev)
    heads = list(range(a.H)) if heads is None else heads
    rows = _rows(a.L, n_rows, a.H)
    for r in ratios:
        k = rmm.rmm_retained_count(r, a.D)
        idx = torch.empty(a.H * k, dtype=torch.int32, device=dev)
        rmm.rmm_select(e, k, idx)
        idx_ref = np.stack([ro.topk_indices(e_ref[h], k) for h in range(a.H)])
        assert check_index_sets(idx.cpu().numpy().reshape(a.H, k), idx_ref, e_ref, a.L) == 0
        rmm.rmm_reduced_qk(Qd, Kd, idx.view(1, a.H, k), S, causal=True)
        # every masked entry of every head is -inf: count per head (any size)
        n_inf = torch.isneginf(S[0]).sum(dim=(1, 2)).cpu().numpy()
        assert np.all(n_inf == a.L * (a.L - 1) // 2)
        Ss = from_device(S[0][:, torch.from_numpy(rows).to(dev)])
        S_ref = ro.reduced_qk(Q, Kc, idx_ref, True, rows=rows)
        for h in heads:
            isclose_inf_pattern(Ss[h], S_ref[h])
            g = ro.gqa_kv_head(h, a.H, a.Hkv)
            I = idx_ref[h]
            absprod = np.abs(Q[h][rows][:, I]).astype(np.float64) @ \
                np.abs(Kc[g][:, I]).astype(np.float64).T
            fin = np.isfinite(S_ref[h])
            check_product(Ss[h][fin], S_ref[h][fin], absprod[fin], k, "bf16",
                          scale=a.D ** -0.5)
    del Qd, Kd, S
    torch.cuda.empty_cache()


def _fused_attention_case(name, ratios, n_rows=11):
    """The reduced attention block at full size: every row's output on
    sampled query rows (first and last included) against the oracle, with
    the index sets from the library's own selection (checked above)."""
    dev = require_gpu()
    wk = wl.WORKLOADS[name]
    a = wk.attention
    q, kk = wl.workload_qk(wk)
    qb, kb = wl.f32_to_bf16_bits(q), wl.f32_to_bf16_bits(kk)
    vb = wl.f32_to_bf16_bits(wl.workload_v(wk))
    Q, Kc, V = wl.decode(qb, "bf16"), wl.decode(kb, "bf16"), wl.decode(vb, "bf16")
    del q, kk
    Qd = _dev_bf16(qb, dev).reshape(1, a.H, a.L, a.D)
    Kd = _dev_bf16(kb, dev).reshape(1, a.Hkv, a.L, a.D)
    Vd = _dev_bf16(vb, dev).reshape(1, a.Hkv, a.L, a.D)
    e_ref = head_energies(Q)
    O = torch.empty((1, a.H, a.L, a.D), dtype=torch.bfloat16, device=dev)
    rows = _rows(a.L, n_rows, a.H + 1)
    Q64, K64, V64 = (x.astype(np.float64) for x in (Q, Kc, V))
    for r in ratios:
        k = rmm.rmm_retained_count(r, a.D)
        idx_ref = np.stack([ro.topk_indices(e_ref[h], k) for h in range(a.H)]).astype(np.int32)
        rmm.rmm_reduced_attention(Qd, Kd, Vd, torch.from_numpy(idx_ref).to(dev).view(1, a.H, k), O,
                                  causal=a.causal)
        Os = from_device(O[0][:, torch.from_numpy(rows).to(dev)])
        ref = ro.reduced_attention(Q64, K64, V64, idx_ref, a.causal, rows=rows)
        bound = attention_bound(Q64, K64, V64, idx_ref, a.causal, a.D ** -0.5, rows=rows)
        err = np.abs(Os - ref)
        assert np.all(err <= bound[:, :, None] + 2.0 ** -8 * np.abs(ref)), float(err.max())
        assert err.max() / max(np.abs(ref).max(), 1e-30) <= NORM_TOL["bf16"]
    del Qd, Kd, Vd, O
    torch.cuda.empty_cache()


RATIOS = (0.25, 0.5, 0.75, 1.0)


@pytest.mark.parametrize("proj", ["gate", "up", "down"])
def test_mlp_1b(proj):
    _projection_case("mlp_1b", proj, RATIOS)


def test_attention_4k():
    _attention_case("attn_4k", RATIOS)


@pytest.mark.parametrize("proj", ["q", "k", "v", "o", "gate", "up", "down"])
def test_layer_8b_projection(proj):
    _projection_case("layer_8b", proj, RATIOS)


def test_layer_8b_attention():
    _attention_case("layer_8b", RATIOS)


def test_layer_8b_fused_attention():
    _fused_attention_case("layer_8b", RATIOS)


def test_attn_4k_fused_attention():
    _fused_attention_case("attn_4k", RATIOS)


# the 70B-class layer on one GPU (16384 tokens, hidden 8192, 64 / 8 heads,
# MLP 28672): every projection, every ratio
@pytest.mark.parametrize("proj", ["q", "k", "v", "o", "gate", "up", "down"])
def test_layer_70b_projection(proj):
    _projection_case("layer_70b", proj, RATIOS)


def test_layer_70b_fused_attention():
    """The reduced attention block on the 70B layer's 64 query / 8 kv heads
    and 16384 tokens, at the outer ratios."""
    _fused_attention_case("layer_70b", (0.25, 1.0), n_rows=5)


def test_layer_70b_attention():
    """Every one of the 64 heads: energies, sets, the -inf count, and
    sampled rows of S against the oracle."""
    _attention_case("layer_70b", RATIOS, n_rows=5)
