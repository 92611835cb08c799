"""Benchmark of the RMM hot path on one MI355X.

One step = one pass of the whole reduced path of an 8B-class decoder layer
(seq 8192, hidden 4096, 32 query / 8 kv heads of dim 128, MLP 14336) at
retention ratio r, on synthetic bf16 inputs already resident in HBM:

  * q/k/v  : energies of the attention input (the scoring pass also writes
             its K-major copy), TopK, one gathered GEMM over the q|k|v weights
             stored concatenated along N (the three projections read one
             input, so they share one set)
  * o      : energies, TopK, gathered GEMM
  * gate/up: energies of the MLP input, TopK, one gathered GEMM (gate|up)
  * down   : energies, TopK, gathered GEMM
  * QK^T   : per-head energies of Q, TopK per head, reduced QK^T (causal)

The headline is retained TFLOP/s (2*M*N*k per projection plus 2*k per
computed causal score) at r = 0.5, with the speedup of the same pipeline
over its own r = 1 run.  Each r is timed separately: W warm-up steps, then
K timed steps bracketed by device synchronisation.

  python bench.py [--gpus 1] [--steps 20] [--warmup 5] [--ratios 0.25,0.5,0.75,1.0]

The same step is also timed under per-component retention ratios
("component_ratios": attention-side products, and optionally the MLP down
projection, at 0.7 with the sensitive gate/up group dense), the policies the
paper's component analysis points to, with the speedup over the r = 1 run.

The fused attention block (softmax of the reduced scores times V, S never
written) is timed on its own after the sweep, at the same ratios, and
reported under "fused_attention" with its speedup over r = 1 and its own
MFMA roofline; it is not part of the step.  "attention_o_chain" times that
block feeding the reduced output projection, with the block writing the
projection's K-major input and column energies (no separate scoring pass)
against the unfused chain; "mlp_chain" likewise for the gate|up GEMM whose
epilogue applies silu(g) * u and writes the down projection's K-major input
and column energies.

A decode step of the same layer (batch 1, one token: energies, TopK and the
reduced product over the retained weight rows per projection group) is timed
the same way and reported under "decode" with its HBM roofline.

The roofline object covers the dominant kernel, the K-major gathered GEMM:
achieved = retained FLOPs of all its timed launches (every ratio of the run)
over their summed durations, taken from HIP events recorded on the stream
the launches go to.  Its HBM traffic per launch comes from rocprofv3 counter
runs of this same command (FETCH_SIZE and WRITE_SIZE, scaled by what the
counters read for a plain device copy of known size, see --copy-probe-mib);
it is reported only while the kernel source is the one those counters
measured.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "reduced-GEMM TFLOP/s (retained FLOPs) + speedup vs dense r=1, 8B shapes, seq 8192"
HEADLINE_R = 0.5
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA, published (no sparsity)
PEAK_HBM_GBS = 8000.0
GEMM_KERNEL = "gemm_kmajor_tr_kernel"
CSRC = os.path.join(ROOT, "paper_2608_13426_amd", "csrc")
BUILD_SCRIPT = os.path.join(ROOT, "paper_2608_13426_amd", "build.py")


def _sources(main):
    """A kernel's translation unit, the headers it includes, and the build
    script (its compiler flags): what the HBM counter figures depend on."""
    return [os.path.join(CSRC, main), os.path.join(CSRC, "device_common.h"),
            os.path.join(CSRC, "kernels.h"), BUILD_SCRIPT]


# HBM bytes per launch (or call) from two rocprofv3 --pmc runs of the default
# ratio mix (FETCH_SIZE x2.0, WRITE_SIZE x1.0: the factors a 512 MiB device
# copy reads), averaged over the kernel's dispatches of the measured command.
# A figure is reported only while the SHA-256 of its sources (the kernel's
# file, the shared headers and the build script) is the one it was measured
# with, and for the same launch mix; re-run the counters after any change.
GEMM_TRAFFIC = {"sources": _sources("gemm.hip"),
                "sha256": "2f2c9f14c1ee2a707e502647b0ed6082ecc70473c4370aa1de688d67103f4f47",
                "mix": "layer_8b r=0.25,0.5,0.75,1.0 grouped",
                "bytes": round((399447.85 * 2.0 + 172169.57) * 1024)}
# per fused attention call: attn_fwd_kernel (mean over the four ratios' kernels)
# plus attn_compact_k_kernel
ATTN_TRAFFIC = {"sources": _sources("attn.hip"),
                "sha256": "2ef66f0b47540990067c3d74bdff9c5089cd7921d90f6202cdc486f4c9858b0d",
                "mix": "layer_8b r=0.25,0.5,0.75,1.0",
                "bytes": round((103628.45 * 2.0 + 65550.75 + 8249.02 * 2.0 + 40960.00) * 1024)}
# per rmm_rmsnorm_kmajor call (8192 x 4096, the same whatever r):
# rms_block_kmajor_kernel and its score_finalize_grouped_kernel
NORM_TRAFFIC = {"sources": _sources("norm.hip") + [os.path.join(CSRC, "score.hip")],
                "sha256": "0340673358c97aa4fbe9598a3ef098cffc971f6775443e358ce25fb38375a34e",
                "mix": "layer_8b attn_in,mlp_in",
                "bytes": round((33033.05 * 2.0 + 74159.67 + 4115.00 * 2.0 + 32.00) * 1024)}

# per rmm_decode_products call of the batch-1 decode step (the four 8B
# groups; mean over the four ratios): gemv_partial_grouped_kernel and
# gemv_reduce_grouped_kernel
DECODE_TRAFFIC = {"sources": [os.path.join(CSRC, f) for f in ("gemv.hip", "kernels.h", "device_common.h")]
                  + [BUILD_SCRIPT],
                  "sha256": "40da861c585557e8e1d6f6498bd11aa8d6d194f9f5d21c30863040a4de695740",
                  "mix": "layer_8b r=0.25,0.5,0.75,1.0 B=1",
                  "bytes": round(((53592.86 * 2.0 + 2661.30 + 1349.0 * 2.0 + 84.0)
                                  + (106951.50 * 2.0 + 3431.99 + 1733.0 * 2.0 + 84.0)
                                  + (160329.72 * 2.0 + 3948.19 + 1993.0 * 2.0 + 84.0)
                                  + (213691.84 * 2.0 + 4222.14 + 2121.0 * 2.0 + 84.0)) / 4 * 1024)}
# per rmm_decode_products_shared call at B = 16, r = 0.5 on the 8B groups:
# its four kernels (boundaries, union pass, product, range reduction)
SHARED_TRAFFIC = {"sources": [os.path.join(CSRC, f) for f in ("gemv_shared.hip", "gemv_shared.h",
                                                              "kernels.h", "device_common.h")]
                  + [BUILD_SCRIPT],
                  "sha256": "7c312c2936bb3855686f59ad095ab0d5a6bfa8657bc397231fe60e4724f12af6",
                  "mix": "layer_8b B=16 r=0.5",
                  "bytes": round((483.0 * 2.0 + 24.5 + 939.6 * 2.0 + 937.6 + 217030.5 * 2.0 + 26646.8
                                  + 13333.0 * 2.0 + 1344.1) * 1024)}


def sources_sha256(paths):
    h = hashlib.sha256()
    for path in paths:
        with open(path, "rb") as f:
            h.update(hashlib.sha256(f.read()).digest())
    return h.hexdigest()


def recorded_traffic(rec, mix):
    """A recorded HBM byte count, if its sources and launch mix are the ones measured."""
    if rec is None or rec["bytes"] is None or rec["mix"] != mix:
        return None
    if sources_sha256(rec["sources"]) != rec["sha256"]:
        return None
    return rec["bytes"]


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--ratios", default="0.25,0.5,0.75,1.0")
    p.add_argument("--workload", default="layer_8b")
    p.add_argument("--cpu-tokens", type=int, default=0,
                   help="tokens of the CPU-oracle sample (default: the whole layer)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-fused-attention", action="store_true",
                   help="skip the separate timing of the fused attention block")
    p.add_argument("--no-decode", action="store_true",
                   help="skip the separate timing of the decode step")
    p.add_argument("--no-decode-batched", action="store_true",
                   help="skip the decode products for batches of sequences (per-sequence, "
                        "shared rows, dense)")
    p.add_argument("--no-attention-chain", action="store_true",
                   help="skip the timing of the attention -> o-projection chain")
    p.add_argument("--no-mlp-chain", action="store_true",
                   help="skip the timing of the MLP chain (fused and unfused)")
    p.add_argument("--no-policies", action="store_true",
                   help="skip the steps with per-component retention ratios")
    p.add_argument("--no-norm-chain", action="store_true",
                   help="skip the timing of the RMSNorm -> projection chains")
    p.add_argument("--no-pv-chain", action="store_true",
                   help="skip the timing of the scores -> weights -> token-axis value product chain")
    p.add_argument("--no-pv", action="store_true",
                   help="skip the separate timing of the token-axis reduced value product")
    p.add_argument("--no-paper-kernels", action="store_true",
                   help="skip the paper's kernel-level benchmark (reduced QK^T and AV at "
                        "L = 1024, 2048, 4096, rho = 0.8)")
    p.add_argument("--no-layer-forward", action="store_true",
                   help="skip the prefill pass of the whole layer (RMM producers and "
                        "products against torch's dense layer)")
    p.add_argument("--copy-probe-mib", type=int, default=0,
                   help="copy this many MiB device to device once before timing (a "
                        "counter-calibration probe for rocprofv3 runs; not timed)")
    return p.parse_args()


# ---------------------------------------------------------------- inputs

def time_decode_batched(L, r, B, steps, warmup):
    """The products of one decode step for B sequences (the first B tokens of
    each input stand in for their current tokens; each sequence's own TopK
    set, made once outside the timed region): rmm_decode_products (each
    sequence reads its own k rows) against rmm_decode_products_shared (each
    row of the union of the B sets read once), and torch's dense product of
    the same B tokens, each as a replayed graph of R back-to-back calls.
    Algorithmic bytes of the shared products: the union rows of every W,
    the tokens and the outputs."""
    import torch
    import paper_2608_13426_amd as rmm
    wk = L.wk
    groups, dense = [], []
    union_bytes = 0
    for name in L.groups:
        K = wk.inputs[name][0]
        k = rmm.rmm_retained_count(ratio_of(r, name), K)
        X = L.X[name][:B].contiguous()
        W = L.Wcat[name]
        N = W.shape[1]
        idx = torch.empty(B * k, dtype=torch.int32, device=L.dev)
        rmm.rmm_select_tokens(X.view(B, 1, K), k, idx)
        groups.append((X, W, k, idx, torch.empty((B, N), dtype=torch.bfloat16, device=L.dev)))
        dense.append((X, W, torch.empty((B, N), dtype=torch.bfloat16, device=L.dev)))
        u = int(np.unique(idx.cpu().numpy()).size)
        union_bytes += u * N * 2 + B * (K + N) * 2 + 4 * B * k
    ws_seq = torch.empty(max(rmm.rmm_decode_step_workspace_size(groups), 1), dtype=torch.uint8,
                         device=L.dev)
    ws_sh = torch.empty(rmm.rmm_decode_products_shared_workspace_size(groups), dtype=torch.uint8,
                        device=L.dev)

    def graph_us(fn, R=10):
        def many():
            for _ in range(R):
                fn()
        g = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            many()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        with torch.cuda.graph(g):
            many()
        for _ in range(warmup):
            g.replay()
        torch.cuda.synchronize()
        start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record()
        for _ in range(steps):
            g.replay()
        end.record()
        torch.cuda.synchronize()
        return start.elapsed_time(end) * 1e3 / (steps * R)

    def dense_fn():
        for X, W, Y in dense:
            torch.matmul(X, W, out=Y)
    seq_us = graph_us(lambda: rmm.rmm_decode_products(groups, workspace=ws_seq))
    sh_us = graph_us(lambda: rmm.rmm_decode_products_shared(groups, workspace=ws_sh))
    d_us = graph_us(dense_fn)
    return {"r": r, "batch": B, "per_sequence_us": seq_us, "shared_us": sh_us, "dense_torch_us": d_us,
            "shared_speedup_vs_per_sequence": seq_us / sh_us, "shared_speedup_vs_dense_torch": d_us / sh_us,
            "union_bytes": union_bytes, "shared_gbs": union_bytes / (sh_us * 1e-6) / 1e9}


class Layer:
    """Device-resident inputs, weights and outputs of one decoder layer."""

    def __init__(self, wk, dev):
        import torch
        import workloads as wl
        self.wk, self.dev = wk, dev
        self.M = wk.M

        def put(f32):
            bits = wl.f32_to_bf16_bits(f32)
            return torch.from_numpy(bits.view(np.int16)).to(dev).view(torch.bfloat16)

        self.X = {name: put(wl.workload_input(wk, name)) for name in wk.inputs}
        # K-major copies written by the scoring pass
        self.Xt = {name: torch.empty((v[0], self.M), dtype=torch.bfloat16, device=dev)
                   for name, v in wk.inputs.items()}
        # groups of projections that read one input (q|k|v, gate|up): their
        # weights are stored concatenated along N, so one GEMM launch per
        # group computes all of them (the same retained rows serve each)
        self.groups = {}
        for p in wk.projections:
            self.groups.setdefault(p.input_name, []).append(p)
        self.Wcat, self.Ycat, self.W, self.Y = {}, {}, {}, {}
        for name, projs in self.groups.items():
            self.Wcat[name] = torch.cat([put(wl.workload_weight(wk, p)) for p in projs], dim=1)
            self.Ycat[name] = torch.empty((self.M, sum(p.N for p in projs)), dtype=torch.bfloat16,
                                          device=dev)
            off = 0
            for p in projs:
                self.W[p.name] = self.Wcat[name][:, off:off + p.N]
                self.Y[p.name] = self.Ycat[name][:, off:off + p.N]
                off += p.N
        a = wk.attention
        q, k = wl.workload_qk(wk)
        self.Q = put(q).reshape(1, a.H, a.L, a.D)
        self.Kc = put(k).reshape(1, a.Hkv, a.L, a.D)
        self.S = torch.empty((1, a.H, a.L, a.L), dtype=torch.bfloat16, device=dev)
        # value rows and output of the fused attention block (timed on its own)
        self.V = put(wl.workload_v(wk)).reshape(1, a.Hkv, a.L, a.D)
        self.O = torch.empty((1, a.H, a.L, a.D), dtype=torch.bfloat16, device=dev)
        Kmax = max(v[0] for v in wk.inputs.values())
        import paper_2608_13426_amd as rmm
        ws = max(rmm.rmm_workspace_size(rmm.RMM_OP_SCORE, 1, self.M, Kmax),
                 rmm.rmm_workspace_size(rmm.RMM_OP_SCORE, a.H, a.L, a.D), 1)
        self.ws = torch.empty(ws, dtype=torch.uint8, device=dev)
        self.energy = torch.empty(max(Kmax, a.H * a.D), dtype=torch.float64, device=dev)
        self.idx = {name: None for name in wk.inputs}
        self.qidx = None


# Component policies (per-component retention ratios; App. B.4, compute-normalized
# component analysis): at RR = 0.7 the attention-side products and the MLP down
# projection lose the least accuracy, the up and gate projections the most, so
# the sensitive group stays dense (r = 1: the same pipeline with k = K).
# Components are the input groups of the step plus "qk" for the per-head QK^T.
POLICIES = {
    "attention_side_0.7": {"attn_in": 0.7, "o_in": 0.7, "qk": 0.7, "mlp_in": 1.0, "down_in": 1.0},
    "attention_side_and_down_0.7": {"attn_in": 0.7, "o_in": 0.7, "qk": 0.7, "mlp_in": 1.0,
                                    "down_in": 0.7},
}


def ratio_of(r, component):
    """The ratio a component runs at: r itself, or its entry in a policy."""
    return r[component] if isinstance(r, dict) else r


def flops(wk, r):
    """Retained FLOPs of one step at ratio r (a float, or a policy dict)."""
    import paper_2608_13426_amd as rmm
    proj = sum(2 * wk.M * p.N * rmm.rmm_retained_count(ratio_of(r, p.input_name), p.K)
               for p in wk.projections)
    a = wk.attention
    pairs = a.L * (a.L + 1) // 2
    qk = 2 * a.H * pairs * rmm.rmm_retained_count(ratio_of(r, "qk"), a.D)
    return proj, qk


def run_step(L, r, gemm_events=None, diag=None):
    """Enqueue one full step on the current stream (r: a ratio or a policy).
    With `diag` (a dict), also record each selection's retained-energy
    fraction (App. B.4: the share of the input's squared norm on the kept
    channels, from the step's own energies and sets; synchronises)."""
    import torch
    import paper_2608_13426_amd as rmm
    wk = L.wk
    for name, projs in L.groups.items():
        K = wk.inputs[name][0]
        k = rmm.rmm_retained_count(ratio_of(r, name), K)
        X = L.X[name]
        e = L.energy[:K]
        rmm.rmm_score_kmajor(X, e, L.Xt[name], L.ws)
        if L.idx[name] is None or L.idx[name].numel() != k:
            L.idx[name] = torch.empty(k, dtype=torch.int32, device=L.dev)
        rmm.rmm_select(e, k, L.idx[name])
        if diag is not None:
            diag[name] = float(e[L.idx[name].long()].sum() / e.sum())
        if gemm_events is not None:
            ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            ev0.record()
        rmm.rmm_reduced_gemm_kmajor(L.Xt[name], L.Wcat[name], L.idx[name].view(1, k), L.Ycat[name])
        if gemm_events is not None:
            ev1.record()
            gemm_events.append((ev0, ev1, 2 * wk.M * L.Ycat[name].shape[1] * k))
    a = wk.attention
    kq = rmm.rmm_retained_count(ratio_of(r, "qk"), a.D)
    e = L.energy[:a.H * a.D]
    rmm.rmm_score(L.Q.reshape(a.H, a.L, a.D), e, L.ws)
    if L.qidx is None or L.qidx.numel() != a.H * kq:
        L.qidx = torch.empty(a.H * kq, dtype=torch.int32, device=L.dev)
    rmm.rmm_select(e, kq, L.qidx)
    if diag is not None:
        eh = e.view(a.H, a.D)
        kept = torch.gather(eh, 1, L.qidx.view(a.H, kq).long()).sum(dim=1)
        diag["qk_heads_mean"] = float((kept / eh.sum(dim=1)).mean())
    rmm.rmm_reduced_qk(L.Q, L.Kc, L.qidx.view(1, a.H, kq), L.S, causal=True)


def time_ratio(L, r, steps, warmup):
    import torch
    for _ in range(warmup):
        run_step(L, r)
    torch.cuda.synchronize()
    events = []
    t0 = time.perf_counter()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        run_step(L, r, gemm_events=events)
    end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = start.elapsed_time(end) / steps
    gemm_ms = sum(a.elapsed_time(b) for a, b, _ in events)
    gemm_flop = sum(f for _, _, f in events)
    proj, qk = flops(L.wk, r)
    diag = {}
    run_step(L, r, diag=diag)                 # untimed: the retained-energy diagnostic
    torch.cuda.synchronize()
    return {
        "r": r, "ms_per_step": ms, "wall_s": wall,
        "tflops": (proj + qk) / (ms * 1e-3) / 1e12,
        "retained_gflop": (proj + qk) / 1e9,
        "gemm_launches": len(events), "gemm_ms_total": gemm_ms, "gemm_gflop_total": gemm_flop / 1e9,
        "gemm_tflops": gemm_flop / (gemm_ms * 1e-3) / 1e12,
        "gemm_avg_us": gemm_ms * 1e3 / max(len(events), 1),
        "gemm_avg_gflop": gemm_flop / max(len(events), 1) / 1e9,
        "retained_energy": {n: round(v, 5) for n, v in diag.items()},
    }


def time_attention(L, r, steps, warmup):
    """The fused reduced attention block on the layer's Q, K, V (causal): the
    per-head selection at ratio r is made once outside the timed region, then
    `steps` calls are timed one by one with HIP events on the launch stream.
    Each call runs the key compaction and the attention kernel; its retained
    FLOPs are 2*H*pairs*(k + D) (reduced scores plus the dense value product)."""
    import torch
    import paper_2608_13426_amd as rmm
    a = L.wk.attention
    kq = rmm.rmm_retained_count(r, a.D)
    e = L.energy[:a.H * a.D]
    rmm.rmm_score(L.Q.reshape(a.H, a.L, a.D), e, L.ws)
    idx = torch.empty(a.H * kq, dtype=torch.int32, device=L.dev)
    rmm.rmm_select(e, kq, idx)
    ws = torch.empty(rmm.rmm_workspace_size(rmm.RMM_OP_ATTENTION, a.H, a.L, a.D, kq),
                     dtype=torch.uint8, device=L.dev)
    args = (L.Q, L.Kc, L.V, idx.view(1, a.H, kq), L.O)
    for _ in range(warmup):
        rmm.rmm_reduced_attention(*args, causal=True, workspace=ws)
    torch.cuda.synchronize()
    evs = []
    for _ in range(steps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        rmm.rmm_reduced_attention(*args, causal=True, workspace=ws)
        e1.record()
        evs.append((e0, e1))
    torch.cuda.synchronize()
    ms = sum(x.elapsed_time(y) for x, y in evs) / steps
    flop = 2 * a.H * (a.L * (a.L + 1) // 2) * (kq + a.D)
    return {"r": r, "k": kq, "avg_call_us": ms * 1e3, "gflop": flop / 1e9,
            "retained_tflops": flop / (ms * 1e-3) / 1e12, "calls": steps}


def time_sdpa(L, steps, warmup):
    """torch's fused causal attention (SDPA limited to its flash and
    memory-efficient kernels, GQA) on the layer's Q, K and V, for context;
    None when neither kernel takes these inputs."""
    import torch
    import torch.nn.functional as F_
    from torch.nn.attention import SDPBackend, sdpa_kernel

    def call():
        with sdpa_kernel([SDPBackend.FLASH_ATTENTION, SDPBackend.EFFICIENT_ATTENTION]):
            return F_.scaled_dot_product_attention(L.Q, L.Kc, L.V, is_causal=True, enable_gqa=True)
    try:
        return time_calls(call, steps, warmup)
    except RuntimeError:
        return None


def time_calls(fn, steps, warmup):
    """Average microseconds of `fn` (launches on the current stream): `warmup`
    untimed calls, then `steps` calls each bracketed by HIP events."""
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    evs = []
    for _ in range(steps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        fn()
        e1.record()
        evs.append((e0, e1))
    torch.cuda.synchronize()
    return sum(x.elapsed_time(y) for x, y in evs) / steps * 1e3


def time_attention_chain(L, r, steps, warmup):
    """The attention block feeding the reduced output projection, both ways,
    at ratio r for the heads' and the projection's selections (the per-head
    selection made once outside the timed region):
      fused   : rmm_reduced_attention_kmajor (writes the projection's K-major
                input and its column energies) -> TopK -> K-major GEMM;
      unfused : rmm_reduced_attention (O per head) -> O laid out as the
                projection's token-major input (a torch copy) ->
                rmm_score_kmajor -> TopK -> K-major GEMM.
    Every call is bracketed by HIP events on the launch stream; the layout
    copy is also timed alone, so the unfused chain can be read without it."""
    import torch
    import paper_2608_13426_amd as rmm
    a, M = L.wk.attention, L.M
    HD = a.H * a.D
    kq = rmm.rmm_retained_count(r, a.D)
    e = L.energy[:HD]
    rmm.rmm_score(L.Q.reshape(a.H, a.L, a.D), e, L.ws)
    idx = torch.empty(a.H * kq, dtype=torch.int32, device=L.dev)
    rmm.rmm_select(e, kq, idx)
    idx = idx.view(1, a.H, kq)
    Wo, Yo = L.W["o"], L.Y["o"]
    ko = rmm.rmm_retained_count(r, HD)
    sel = torch.empty(ko, dtype=torch.int32, device=L.dev)
    ws_k = torch.empty(rmm.rmm_attention_kmajor_workspace_size(1, a.H, a.L, a.L, a.D, kq),
                       dtype=torch.uint8, device=L.dev)
    ws_a = torch.empty(rmm.rmm_workspace_size(rmm.RMM_OP_ATTENTION, a.H, a.L, a.D, kq),
                       dtype=torch.uint8, device=L.dev)
    Ot = torch.empty((HD, a.L), dtype=torch.bfloat16, device=L.dev)
    Xo = torch.empty((a.L, HD), dtype=torch.bfloat16, device=L.dev)
    Xt = L.Xt["o_in"]
    eo = torch.empty(HD, dtype=torch.float64, device=L.dev)

    def fused():
        rmm.rmm_reduced_attention_kmajor(L.Q, L.Kc, L.V, idx, Ot, eo, causal=True, workspace=ws_k)
        rmm.rmm_select(eo, ko, sel)
        rmm.rmm_reduced_gemm_kmajor(Ot, Wo, sel.view(1, ko), Yo)

    def layout():
        Xo.view(a.L, a.H, a.D).copy_(L.O[0].permute(1, 0, 2))

    def unfused():
        rmm.rmm_reduced_attention(L.Q, L.Kc, L.V, idx, L.O, causal=True, workspace=ws_a)
        layout()
        rmm.rmm_score_kmajor(Xo, eo, Xt, L.ws)
        rmm.rmm_select(eo, ko, sel)
        rmm.rmm_reduced_gemm_kmajor(Xt, Wo, sel.view(1, ko), Yo)

    us_f, us_u, us_l = (time_calls(f, steps, warmup) for f in (fused, unfused, layout))
    return {"r": r, "k_heads": kq, "k_o": ko, "fused_us": us_f, "unfused_us": us_u,
            "layout_copy_us": us_l, "unfused_without_copy_us": us_u - us_l,
            "speedup": us_u / us_f, "speedup_without_copy": (us_u - us_l) / us_f, "calls": steps}


def time_mlp_chain(L, r, steps, warmup):
    """The MLP of the layer at ratio r (both selections), both ways:
      fused   : energies + TopK of the MLP input -> rmm_reduced_gemm_swiglu_kmajor
                (the gate|up product whose epilogue writes the down
                projection's K-major input H^T and its column energies) ->
                TopK -> down K-major GEMM;
      unfused : energies + TopK -> gate|up GEMM (Y) -> torch silu(g) * u (H,
                token-major) -> rmm_score_kmajor(H) -> TopK -> down GEMM.
    Every call is bracketed by HIP events on the launch stream; the torch
    activation is also timed alone."""
    import torch
    import paper_2608_13426_amd as rmm
    wk, M = L.wk, L.M
    K = wk.inputs["mlp_in"][0]
    F = wk.inputs["down_in"][0]
    k = rmm.rmm_retained_count(r, K)
    kd = rmm.rmm_retained_count(r, F)
    idx = torch.empty(k, dtype=torch.int32, device=L.dev)
    sel = torch.empty(kd, dtype=torch.int32, device=L.dev)
    Wgu = rmm.swiglu_weight_layout(L.W["gate"], L.W["up"])
    Ht = torch.empty((F, M), dtype=torch.bfloat16, device=L.dev)
    H = torch.empty((M, F), dtype=torch.bfloat16, device=L.dev)
    eh = torch.empty(F, dtype=torch.float64, device=L.dev)
    ws_s = torch.empty(rmm.rmm_gemm_swiglu_workspace_size(1, M, F), dtype=torch.uint8,
                       device=L.dev)
    X, Xt, e = L.X["mlp_in"], L.Xt["mlp_in"], L.energy[:K]
    Xtd, Wd, Yd, Ygu = L.Xt["down_in"], L.W["down"], L.Y["down"], L.Ycat["mlp_in"]

    def head():
        rmm.rmm_score_kmajor(X, e, Xt, L.ws)
        rmm.rmm_select(e, k, idx)

    def fused():
        head()
        rmm.rmm_reduced_gemm_swiglu_kmajor(Xt, Wgu, idx.view(1, k), Ht, eh, workspace=ws_s)
        rmm.rmm_select(eh, kd, sel)
        rmm.rmm_reduced_gemm_kmajor(Ht, Wd, sel.view(1, kd), Yd)

    def activation():
        torch.mul(torch.nn.functional.silu(Ygu[:, :F]), Ygu[:, F:], out=H)

    def unfused():
        head()
        rmm.rmm_reduced_gemm_kmajor(Xt, L.Wcat["mlp_in"], idx.view(1, k), Ygu)
        activation()
        rmm.rmm_score_kmajor(H, eh, Xtd, L.ws)
        rmm.rmm_select(eh, kd, sel)
        rmm.rmm_reduced_gemm_kmajor(Xtd, Wd, sel.view(1, kd), Yd)

    us_f, us_u, us_a = (time_calls(f, steps, warmup) for f in (fused, unfused, activation))
    flop = 2 * M * (2 * F) * k + 2 * M * wk.inputs["mlp_in"][0] * kd
    return {"r": r, "k_gate_up": k, "k_down": kd, "fused_us": us_f, "unfused_us": us_u,
            "activation_us": us_a, "unfused_without_activation_us": us_u - us_a,
            "speedup": us_u / us_f, "speedup_without_activation": (us_u - us_a) / us_f,
            "retained_tflops_fused": flop / (us_f * 1e-6) / 1e12, "calls": steps}


def time_norm_chain(L, name, r, steps, warmup, eps=1e-5):
    """The normalisation in front of a projection group (attn_in: q|k|v,
    mlp_in: gate|up) feeding its reduced GEMM at ratio r, both ways, with the
    layer's activations standing in for the pre-norm hidden state:
      fused   : rmm_rmsnorm_kmajor (one pass over X: the normalised rows
                K-major and their column energies) -> TopK -> K-major GEMM;
      unfused : torch RMSNorm (row-major normalised rows) -> rmm_score_kmajor
                -> TopK -> K-major GEMM.
    Every call is bracketed by HIP events; the producer alone and the torch
    normalisation alone are timed too."""
    import torch
    import paper_2608_13426_amd as rmm
    import workloads as wl
    wk, M = L.wk, L.M
    K = wk.inputs[name][0]
    k = rmm.rmm_retained_count(r, K)
    X, Xt, e = L.X[name], L.Xt[name], L.energy[:K]
    g = torch.from_numpy(wl.f32_to_bf16_bits(1.0 + 0.3 * wl.normal_blocks((wk.seed, 77), (1, K))[0])
                         .view(np.int16)).to(L.dev).view(torch.bfloat16)
    idx = torch.empty(k, dtype=torch.int32, device=L.dev)
    Y = torch.empty((M, K), dtype=torch.bfloat16, device=L.dev)
    ws_n = torch.empty(rmm.rmm_rmsnorm_kmajor_workspace_size(1, M, K), dtype=torch.uint8,
                       device=L.dev)
    W, Yo = L.Wcat[name], L.Ycat[name]

    def producer():
        rmm.rmm_rmsnorm_kmajor(X, g, eps, Xt.view(1, K, M), e, ws_n)

    def torch_norm():
        xf = X.float()
        t = (xf * torch.rsqrt(xf.pow(2).mean(dim=-1, keepdim=True) + eps)).to(torch.bfloat16)
        torch.mul(t, g, out=Y)

    def score():
        rmm.rmm_score_kmajor(Y, e, Xt, L.ws)

    def tail():
        rmm.rmm_select(e, k, idx)
        rmm.rmm_reduced_gemm_kmajor(Xt, W, idx.view(1, k), Yo)

    def fused():
        producer()
        tail()

    def unfused():
        torch_norm()
        score()
        tail()

    us = {n: time_calls(f, steps, warmup) for n, f in
          (("fused", fused), ("unfused", unfused), ("producer", producer),
           ("torch_norm", torch_norm), ("score_kmajor", score))}
    nbytes = 2 * M * K * 2 + 8 * K           # read X, write Xt, energies
    return {"input": name, "r": r, "K": K, "k": k, "fused_us": us["fused"],
            "unfused_us": us["unfused"], "producer_us": us["producer"],
            "torch_norm_us": us["torch_norm"], "score_kmajor_us": us["score_kmajor"],
            "unfused_without_norm_us": us["unfused"] - us["torch_norm"],
            "speedup": us["unfused"] / us["fused"],
            "speedup_without_norm": (us["unfused"] - us["torch_norm"]) / us["fused"],
            "producer_bytes": nbytes, "producer_gbs": nbytes / (us["producer"] * 1e-6) / 1e9,
            "calls": steps}


def time_pv_chain(L, r, steps, warmup, bufs):
    """The value product fed by its producer, on the layer's causal scores S
    (those of the headline ratio: per head the reduced QK^T over k = 64 of
    the 128 dims) and values V:
      reduced : rmm_attention_weights_kmajor (softmax weights written K-major
                with their token energies; the masked half of S is never
                read) -> TopK of the token energies per head ->
                rmm_reduced_pv_kmajor (kept token rows, causal row tiles
                stopped at their last visible token);
      dense   : torch softmax of S (row-major weights) -> torch P @ V (V
                repeated over each kv head's query heads).
    From the scores' producer on, two ways (S rewritten with the same
    values by the layer's own selection):
      from_qk          : rmm_reduced_qk -> the reduced chain above;
      from_qk_rowstats : rmm_reduced_qk_rowstats (S with its softmax row
                         statistics) -> rmm_attention_weights_kmajor_rowstats
                         (S read once) -> TopK -> rmm_reduced_pv_kmajor.
    Every call is bracketed by HIP events; the producers and the product are
    also timed alone."""
    import torch
    import paper_2608_13426_amd as rmm
    a = L.wk.attention
    kt = rmm.rmm_retained_count(r, a.L)
    Pt, e, ws, P, Vr = bufs["Pt"], bufs["e"], bufs["ws"], bufs["P"], bufs["Vr"]
    rmax, rinv = bufs["rmax"], bufs["rinv"]
    idx = torch.empty(a.H * kt, dtype=torch.int32, device=L.dev)
    kq = L.qidx.numel() // a.H
    qidx = L.qidx.view(1, a.H, kq)

    def producer():
        rmm.rmm_attention_weights_kmajor(L.S, Pt, e, causal=True, workspace=ws)

    def product():
        rmm.rmm_reduced_pv_kmajor(Pt, L.V, idx.view(a.H, kt), L.O, causal=True)

    def reduced():
        producer()
        rmm.rmm_select(e, kt, idx)
        product()

    def dense():
        torch.softmax(L.S[0], dim=-1, out=P)
        torch.matmul(P, Vr, out=bufs["Od"])

    def qk():
        rmm.rmm_reduced_qk(L.Q, L.Kc, qidx, L.S, causal=True)

    def qk_rowstats():
        rmm.rmm_reduced_qk_rowstats(L.Q, L.Kc, qidx, L.S, rmax, rinv, causal=True)

    def producer_rowstats():
        rmm.rmm_attention_weights_kmajor(L.S, Pt, e, causal=True, workspace=ws, row_max=rmax,
                                         row_rinv=rinv)

    def from_qk():
        qk()
        reduced()

    def from_qk_rowstats():
        qk_rowstats()
        producer_rowstats()
        rmm.rmm_select(e, kt, idx)
        product()

    us = {n: time_calls(f, steps, warmup) for n, f in
          (("reduced", reduced), ("producer", producer), ("product", product),
           ("from_qk", from_qk), ("from_qk_rowstats", from_qk_rowstats))}
    if bufs.get("qk_us") is None:
        bufs["qk_us"] = time_calls(qk, steps, warmup)
        bufs["qk_rowstats_us"] = time_calls(qk_rowstats, steps, warmup)
        bufs["producer_rowstats_us"] = time_calls(producer_rowstats, steps, warmup)
    # bytes of the producer: the causal part of S read once, the part of Pt
    # it stores (the lower triangle and, above the diagonal, the zeros of the
    # 256-query block holding each column's diagonal), the energies
    pairs = a.L * (a.L + 1) // 2
    stored = sum(a.L - 256 * (t // 256) for t in range(a.L))
    nbytes = a.H * (pairs * 2 + stored * 2 + a.L * 8)
    rec = {"r": r, "kt": kt, "reduced_us": us["reduced"], "producer_us": us["producer"],
           "product_us": us["product"], "producer_bytes": nbytes,
           "producer_gbs": nbytes / (us["producer"] * 1e-6) / 1e9,
           "qk_k": kq, "qk_us": bufs["qk_us"], "qk_rowstats_us": bufs["qk_rowstats_us"],
           "producer_rowstats_us": bufs["producer_rowstats_us"],
           "producer_rowstats_gbs": nbytes / (bufs["producer_rowstats_us"] * 1e-6) / 1e9,
           "from_qk_us": us["from_qk"], "from_qk_rowstats_us": us["from_qk_rowstats"],
           "rowstats_speedup": us["from_qk"] / us["from_qk_rowstats"], "calls": steps}
    if bufs.get("dense_us") is None:
        bufs["dense_us"] = time_calls(dense, steps, warmup)
    rec["dense_torch_us"] = bufs["dense_us"]
    rec["speedup_vs_dense_torch"] = bufs["dense_us"] / us["reduced"]
    return rec


def attention_weights(L):
    """P = softmax(S) per head, in place in L.S (bf16).  S holds the causal
    scores of the headline ratio (one untimed step at r = 0.5 leaves them
    there: per head the reduced QK^T over 64 of the 128 dims, scaled), so P
    is the layer's attention weights (masked entries -inf -> weight 0)."""
    import torch
    a = L.wk.attention
    for h in range(a.H):
        L.S[0, h] = torch.softmax(L.S[0, h].float(), dim=-1).to(torch.bfloat16)
    torch.cuda.synchronize()


def time_pv(L, r, steps, warmup, ws):
    """The token-axis reduced value product on the layer's attention weights
    P (L.S after attention_weights) and values V: per query head the TopK of
    the column norms of P, then P[:, T] V[T, :] (rmm_reduced_pv: scoring with
    the K-major copy of P, TopK, one gathered product per kv head), timed call
    by call with HIP events; and torch's dense bf16 product P @ V (V repeated
    over each kv head's query heads) for reference."""
    import torch
    import paper_2608_13426_amd as rmm
    a = L.wk.attention
    kt = rmm.rmm_retained_count(r, a.L)
    idx = torch.empty(a.H * kt, dtype=torch.int32, device=L.dev)

    def call():
        rmm.rmm_reduced_pv(L.S, L.V, kt, L.O, idx_out=idx, workspace=ws)

    for _ in range(warmup):
        call()
    torch.cuda.synchronize()
    evs = []
    for _ in range(steps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        call()
        e1.record()
        evs.append((e0, e1))
    torch.cuda.synchronize()
    ms = sum(x.elapsed_time(y) for x, y in evs) / steps
    flop = 2 * a.H * a.L * kt * a.D
    # one read of P (the least any evaluation of the token scores moves), the
    # kept value rows, and O
    nbytes = a.H * a.L * a.L * 2 + a.Hkv * kt * a.D * 2 + a.H * a.L * a.D * 2
    return {"r": r, "kt": kt, "avg_call_us": ms * 1e3, "gflop": flop / 1e9,
            "retained_tflops": flop / (ms * 1e-3) / 1e12, "bytes": nbytes,
            "gbs": nbytes / (ms * 1e-3) / 1e9, "calls": steps}


def time_dense_pv(L, steps, warmup):
    import torch
    a = L.wk.attention
    Vr = L.V.repeat_interleave(a.H // a.Hkv, dim=1).contiguous()
    out = torch.empty_like(L.O)
    for _ in range(warmup):
        torch.matmul(L.S, Vr, out=out)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        torch.matmul(L.S, Vr, out=out)
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e3 / steps


def time_decode(L, r, steps, warmup, B=1):
    """One decode step of the layer's projections for B sequences (one token
    each: the first B tokens of each input stand in for the current tokens):
    per input group, the TopK of the token's squared activations
    (rmm_select_tokens: the same set as energies + TopK for one row) and the
    reduced product that reads only the retained weight rows
    (rmm_reduced_gemv).  The whole step is timed with HIP events (eager and
    as one replayed graph); the step's products alone (rmm_decode_products
    over its sets: the grouped product and reduction launches) are timed as a
    replayed graph of R back-to-back calls, so no host launch gap enters
    their roofline."""
    import torch
    import paper_2608_13426_amd as rmm
    wk = L.wk
    parts = []
    for name in L.groups:
        K = wk.inputs[name][0]
        k = rmm.rmm_retained_count(ratio_of(r, name), K)
        X = L.X[name][:B].reshape(B, 1, K)
        W = L.Wcat[name]
        N = W.shape[1]
        gws = torch.empty(max(rmm.rmm_gemv_workspace_size(B, 1, N, k), 1), dtype=torch.uint8,
                          device=L.dev)
        parts.append({"X": X, "W": W, "k": k, "K": K, "N": N, "ws": gws,
                      "idx": torch.empty(B * k, dtype=torch.int32, device=L.dev),
                      "Y": torch.empty((B, 1, N), dtype=torch.bfloat16, device=L.dev)})

    def step():
        for p in parts:
            rmm.rmm_select_tokens(p["X"], p["k"], p["idx"])
            rmm.rmm_reduced_gemv(p["X"], p["W"], p["idx"].view(B, p["k"]), p["Y"], workspace=p["ws"])

    # the same step as one grouped call: selection, products and slice
    # reductions of the four groups in three launches
    groups = [(p["X"].view(B, p["K"]), p["W"], p["k"], p["idx"], p["Y"].view(B, p["N"])) for p in parts]
    gws = torch.empty(max(rmm.rmm_decode_step_workspace_size(groups), 1), dtype=torch.uint8,
                      device=L.dev)

    def grouped():
        rmm.rmm_decode_step(groups, workspace=gws)

    def captured(fn):
        g = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            fn()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        with torch.cuda.graph(g):
            fn()
        return g

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        step()
    end.record()
    torch.cuda.synchronize()
    us_eager = start.elapsed_time(end) * 1e3 / steps
    # a serving loop replays the step as one HIP graph (every call here is
    # capturable: no allocation, no memset, no synchronisation)
    graph = captured(step)
    for _ in range(warmup):
        graph.replay()
    torch.cuda.synchronize()
    start.record()
    for _ in range(steps):
        graph.replay()
    end.record()
    torch.cuda.synchronize()
    us_sep = start.elapsed_time(end) * 1e3 / steps
    for _ in range(warmup):
        grouped()
    torch.cuda.synchronize()
    start.record()
    for _ in range(steps):
        grouped()
    end.record()
    torch.cuda.synchronize()
    us_grouped_eager = start.elapsed_time(end) * 1e3 / steps
    ggraph = captured(grouped)
    for _ in range(warmup):
        ggraph.replay()
    torch.cuda.synchronize()
    start.record()
    for _ in range(steps):
        ggraph.replay()
    end.record()
    torch.cuda.synchronize()
    us = start.elapsed_time(end) * 1e3 / steps
    # the step's products alone (rmm_decode_products over the sets the step
    # just made: the same two launches), R back-to-back calls per replay
    R = 10

    def products():
        for _ in range(R):
            rmm.rmm_decode_products(groups, workspace=gws)
    pg = captured(products)
    for _ in range(warmup):
        pg.replay()
    torch.cuda.synchronize()
    start.record()
    for _ in range(steps):
        pg.replay()
    end.record()
    torch.cuda.synchronize()
    g_us = start.elapsed_time(end) * 1e3 / (steps * R)
    g_bytes = sum(B * p["k"] * p["N"] * 2 + B * (p["K"] + p["N"]) * 2 + 4 * B * p["k"] for p in parts)
    return {"r": r, "batch": B, "us_per_step": min(us, us_grouped_eager), "us_per_step_grouped_graph": us,
            "us_per_step_grouped_eager": us_grouped_eager,
            "us_per_step_separate": us_sep, "us_per_step_separate_eager": us_eager,
            "gemv_groups_per_call": len(parts),
            "gemv_us_per_step": g_us, "gemv_bytes_per_step": g_bytes,
            "gemv_gbs": g_bytes / (g_us * 1e-6) / 1e9}


def time_layer_forward(L, steps, warmup, ratios=(0.5, 0.8, 1.0), eps=1e-5):
    """One prefill pass of the whole decoder layer (batch 1, the layer's
    attention input standing in for its hidden state x; rotary position
    embedding left out on both sides), every product reduced at ratio r and
    every reduced input produced K-major with its energies by its producer:
      h1 = x + o-proj(attention(q|k|v-proj(rmsnorm(x))))
      h2 = h1 + down(swiglu(gate|up(rmsnorm(h1))))
    as rmm_rmsnorm_kmajor -> TopK -> q|k|v GEMM -> heads laid out (torch
    copies) -> per-head scoring + TopK -> rmm_reduced_attention_kmajor -> TopK
    -> o GEMM -> residual (torch) -> rmm_rmsnorm_kmajor -> TopK ->
    rmm_reduced_gemm_swiglu_kmajor -> TopK -> down GEMM -> residual (torch);
    against torch's dense layer (RMSNorm in fp32, x @ W products, SDPA with
    its fused flash or memory-efficient kernels only, silu(g) * u).  Every
    pass is bracketed by HIP events.  rel_diff_vs_torch: ||h2 - h2_torch|| /
    ||h2_torch|| for the pass at that ratio (at r = 1 only rounding differs)."""
    import torch
    import torch.nn.functional as F_
    import paper_2608_13426_amd as rmm
    import workloads as wl
    wk, M, dev = L.wk, L.M, L.dev
    a = wk.attention
    HD, KVD = a.H * a.D, a.Hkv * a.D
    Dm = wk.inputs["attn_in"][0]
    Fh = wk.inputs["down_in"][0]
    bf = lambda t: t.to(torch.bfloat16)
    gam = [bf(torch.from_numpy(1.0 + 0.3 * wl.normal_blocks((wk.seed, 77 + i), (1, Dm))[0]).to(dev))
           for i in range(2)]
    x = L.X["attn_in"]
    Wqkv, Wo, Wd = L.Wcat["attn_in"], L.Wcat["o_in"], L.Wcat["down_in"]
    Wgu_cat = L.Wcat["mlp_in"]
    Wgu = rmm.swiglu_weight_layout(L.W["gate"], L.W["up"])
    # RMM path buffers
    Xt_a = torch.empty((Dm, M), dtype=torch.bfloat16, device=dev)
    Xt_m = torch.empty_like(Xt_a)
    e_n = torch.empty(Dm, dtype=torch.float64, device=dev)
    ws_n = torch.empty(rmm.rmm_rmsnorm_kmajor_workspace_size(1, M, Dm), dtype=torch.uint8, device=dev)
    Yqkv = torch.empty((M, Wqkv.shape[1]), dtype=torch.bfloat16, device=dev)
    Q = torch.empty((1, a.H, M, a.D), dtype=torch.bfloat16, device=dev)
    Kh = torch.empty((1, a.Hkv, M, a.D), dtype=torch.bfloat16, device=dev)
    Vh = torch.empty_like(Kh)
    e_q = torch.empty(a.H * a.D, dtype=torch.float64, device=dev)
    ws_q = torch.empty(max(rmm.rmm_workspace_size(rmm.RMM_OP_SCORE, a.H, M, a.D), 1), dtype=torch.uint8,
                       device=dev)
    Ot = torch.empty((HD, M), dtype=torch.bfloat16, device=dev)
    e_o = torch.empty(HD, dtype=torch.float64, device=dev)
    Yo = torch.empty((M, Wo.shape[1]), dtype=torch.bfloat16, device=dev)
    h1 = torch.empty_like(x)
    Ht = torch.empty((Fh, M), dtype=torch.bfloat16, device=dev)
    e_h = torch.empty(Fh, dtype=torch.float64, device=dev)
    ws_s = torch.empty(rmm.rmm_gemm_swiglu_workspace_size(1, M, Fh), dtype=torch.uint8, device=dev)
    Yd = torch.empty((M, Wd.shape[1]), dtype=torch.bfloat16, device=dev)
    h2 = torch.empty_like(x)
    rec = {}
    outs = {}
    for r in ratios:
        k_in = rmm.rmm_retained_count(r, Dm)
        k_q = rmm.rmm_retained_count(r, a.D)
        k_o = rmm.rmm_retained_count(r, HD)
        k_d = rmm.rmm_retained_count(r, Fh)
        i_a = torch.empty(k_in, dtype=torch.int32, device=dev)
        i_m = torch.empty_like(i_a)
        i_q = torch.empty(a.H * k_q, dtype=torch.int32, device=dev)
        i_o = torch.empty(k_o, dtype=torch.int32, device=dev)
        i_d = torch.empty(k_d, dtype=torch.int32, device=dev)
        ws_k = torch.empty(rmm.rmm_attention_kmajor_workspace_size(1, a.H, M, M, a.D, k_q),
                           dtype=torch.uint8, device=dev)

        def layer():
            rmm.rmm_rmsnorm_kmajor(x, gam[0], eps, Xt_a, e_n, ws_n)
            rmm.rmm_select(e_n, k_in, i_a)
            rmm.rmm_reduced_gemm_kmajor(Xt_a, Wqkv, i_a.view(1, k_in), Yqkv)
            Q[0].copy_(Yqkv[:, :HD].view(M, a.H, a.D).transpose(0, 1))
            Kh[0].copy_(Yqkv[:, HD:HD + KVD].view(M, a.Hkv, a.D).transpose(0, 1))
            Vh[0].copy_(Yqkv[:, HD + KVD:].view(M, a.Hkv, a.D).transpose(0, 1))
            rmm.rmm_score(Q.reshape(a.H, M, a.D), e_q, ws_q)
            rmm.rmm_select(e_q, k_q, i_q)
            rmm.rmm_reduced_attention_kmajor(Q, Kh, Vh, i_q.view(1, a.H, k_q), Ot, e_o, causal=True,
                                             workspace=ws_k)
            rmm.rmm_select(e_o, k_o, i_o)
            rmm.rmm_reduced_gemm_kmajor(Ot, Wo, i_o.view(1, k_o), Yo)
            torch.add(x, Yo, out=h1)
            rmm.rmm_rmsnorm_kmajor(h1, gam[1], eps, Xt_m, e_n, ws_n)
            rmm.rmm_select(e_n, k_in, i_m)
            rmm.rmm_reduced_gemm_swiglu_kmajor(Xt_m, Wgu, i_m.view(1, k_in), Ht, e_h, workspace=ws_s)
            rmm.rmm_select(e_h, k_d, i_d)
            rmm.rmm_reduced_gemm_kmajor(Ht, Wd, i_d.view(1, k_d), Yd)
            torch.add(h1, Yd, out=h2)
        rec[f"rmm_ms@{r}"] = time_calls(layer, steps, warmup) / 1e3
        layer()
        outs[r] = h2.float().clone()
        del ws_k

    from torch.nn.attention import SDPBackend, sdpa_kernel

    def rmsnorm(t, g):
        tf = t.float()
        return bf(bf(tf * torch.rsqrt(tf.pow(2).mean(-1, keepdim=True) + eps)).float() * g.float())

    def dense():
        qkv = rmsnorm(x, gam[0]) @ Wqkv
        q = qkv[:, :HD].view(M, a.H, a.D).transpose(0, 1)[None]
        kk = qkv[:, HD:HD + KVD].view(M, a.Hkv, a.D).transpose(0, 1)[None]
        vv = qkv[:, HD + KVD:].view(M, a.Hkv, a.D).transpose(0, 1)[None]
        with sdpa_kernel([SDPBackend.FLASH_ATTENTION, SDPBackend.EFFICIENT_ATTENTION]):
            att = F_.scaled_dot_product_attention(q, kk, vv, is_causal=True, enable_gqa=True)
        d1 = x + att[0].transpose(0, 1).reshape(M, HD) @ Wo
        gu = rmsnorm(d1, gam[1]) @ Wgu_cat
        hh = F_.silu(gu[:, :Fh]) * gu[:, Fh:]
        return d1 + hh @ Wd
    try:
        rec["torch_dense_ms"] = time_calls(dense, steps, warmup) / 1e3
        ref = dense().float()
        for r in ratios:
            rec[f"rel_diff_vs_torch@{r}"] = float((outs[r] - ref).norm() / ref.norm())
            rec[f"speedup_vs_torch@{r}"] = rec["torch_dense_ms"] / rec[f"rmm_ms@{r}"]
    except RuntimeError as err:              # no fused SDPA kernel for these inputs
        rec["torch_dense_ms"] = None
        rec["torch_dense_error"] = str(err)[:200]
    for r in ratios:
        rec[f"speedup_vs_r1@{r}"] = rec["rmm_ms@1.0"] / rec[f"rmm_ms@{r}"] if "rmm_ms@1.0" in rec else None
    return {kk: (round(v, 4) if isinstance(v, float) else v) for kk, v in rec.items()}


# The paper's kernel-level latency table (Sec. 6, "GEMM kernel latency"):
# LLaMA-3.1-8B attention, batch 1, rho = 0.8, each RMM operation timed with
# its scoring and TopK; dense and RMM milliseconds on an A100 (context only).
PAPER_A100_MS = {
    ("qk", 1024): (0.120, 0.089), ("qk", 2048): (0.433, 0.336), ("qk", 4096): (1.675, 1.071),
    ("av", 1024): (0.065, 0.039), ("av", 2048): (0.207, 0.114), ("av", 4096): (0.753, 0.399),
}


def time_paper_kernels(wk, dev, steps, warmup, rho=0.8, lengths=(1024, 2048, 4096)):
    """The paper's kernel-level benchmark on this GPU: per sequence length L
    (32 query / 8 kv heads, d = 128, causal, batch 1, the 8B layer's Q, K and
    V recipe cut to L tokens), at retention rho and at 1:
      qk       : rmm_score of Q per head -> rmm_select -> rmm_reduced_qk (S
                 written, masked), against torch's dense bf16 Q @ K^T (K
                 repeated over each kv head's query heads, transposed once
                 outside the timed region);
      av       : rmm_reduced_pv on the row-major weights P (column norms of P
                 -> TopK -> gathered product), against torch's dense P @ V;
      av_chain : from the scores S, rmm_attention_weights_kmajor (weights
                 K-major with their token energies) -> rmm_select ->
                 rmm_reduced_pv_kmajor, against torch softmax + P @ V.
    S holds the full causal scores (the qk pipeline at r = 1) and P their
    softmax (untimed).  Every call is bracketed by HIP events."""
    import torch
    import paper_2608_13426_amd as rmm
    import workloads as wl
    a = wk.attention
    H, Hkv, D, G = a.H, a.Hkv, a.D, a.H // a.Hkv
    out = {}
    for Ln in lengths:
        qf, kf = wl.workload_qk(wk, Ln)
        vf = wl.workload_v(wk, Ln)
        bf = lambda x: torch.from_numpy(wl.f32_to_bf16_bits(x).view(np.int16)).to(dev).view(torch.bfloat16)
        Q, Kc, V = bf(qf)[None], bf(kf)[None], bf(vf)[None]
        S = torch.empty((1, H, Ln, Ln), dtype=torch.bfloat16, device=dev)
        P = torch.empty_like(S)
        O = torch.empty((1, H, Ln, D), dtype=torch.bfloat16, device=dev)
        e = torch.empty(H * max(D, Ln), dtype=torch.float64, device=dev)
        ws = torch.empty(max(rmm.rmm_workspace_size(rmm.RMM_OP_SCORE, H, Ln, D, D), 1),
                         dtype=torch.uint8, device=dev)
        rec = {"L": Ln}
        for r in (rho, 1.0):           # S ends as the full causal scores
            k = rmm.rmm_retained_count(r, D)
            idx = torch.empty(H * k, dtype=torch.int32, device=dev)

            def qk():
                rmm.rmm_score(Q.reshape(H, Ln, D), e[:H * D], ws)
                rmm.rmm_select(e[:H * D], k, idx)
                rmm.rmm_reduced_qk(Q, Kc, idx.view(1, H, k), S, causal=True)
            rec[f"qk_rmm_us@{r}"] = time_calls(qk, steps, warmup)
        Kt = Kc.repeat_interleave(G, dim=1).transpose(-1, -2).contiguous()
        rec["qk_dense_torch_us"] = time_calls(lambda: torch.matmul(Q, Kt, out=P), steps, warmup)
        del Kt
        Vr = V.repeat_interleave(G, dim=1).contiguous()
        Pt = torch.empty_like(S)
        wsw = torch.empty(rmm.rmm_attention_weights_kmajor_workspace_size(1, H, Ln, Ln),
                          dtype=torch.uint8, device=dev)
        for r in (rho, 1.0):
            kt = rmm.rmm_retained_count(r, Ln)
            idt = torch.empty(H * kt, dtype=torch.int32, device=dev)

            def chain():
                rmm.rmm_attention_weights_kmajor(S, Pt, e[:H * Ln], causal=True, workspace=wsw)
                rmm.rmm_select(e[:H * Ln], kt, idt)
                rmm.rmm_reduced_pv_kmajor(Pt, V, idt.view(H, kt), O, causal=True)
            rec[f"av_chain_rmm_us@{r}"] = time_calls(chain, steps, warmup)

        def dense_chain():
            torch.softmax(S[0], dim=-1, out=P[0])
            torch.matmul(P, Vr, out=O)
        rec["av_chain_dense_torch_us"] = time_calls(dense_chain, steps, warmup)
        del Pt, wsw
        # P = the softmax weights, row-major (left by the dense chain)
        wpv = torch.empty(max(rmm.rmm_workspace_size(rmm.RMM_OP_PV, H, Ln, Ln, Ln), 1),
                          dtype=torch.uint8, device=dev)
        for r in (rho, 1.0):
            kt = rmm.rmm_retained_count(r, Ln)
            rec[f"av_rmm_us@{r}"] = time_calls(lambda: rmm.rmm_reduced_pv(P, V, kt, O, workspace=wpv),
                                               steps, warmup)
        rec["av_dense_torch_us"] = time_calls(lambda: torch.matmul(P, Vr, out=O), steps, warmup)
        for op in ("qk", "av", "av_chain"):
            rec[f"{op}_speedup_vs_dense_torch"] = rec[f"{op}_dense_torch_us"] / rec[f"{op}_rmm_us@{rho}"]
            rec[f"{op}_speedup_vs_r1"] = rec[f"{op}_rmm_us@1.0"] / rec[f"{op}_rmm_us@{rho}"]
        for op in ("qk", "av"):
            d_ms, r_ms = PAPER_A100_MS[(op, Ln)]
            rec[f"{op}_paper_a100_ms"] = {"dense": d_ms, "rmm": r_ms, "speedup": round(d_ms / r_ms, 2)}
        out[Ln] = {kk: (round(v, 3) if isinstance(v, float) else v) for kk, v in rec.items()}
        del Q, Kc, V, S, P, O, Vr, wpv
        torch.cuda.empty_cache()
    return out


# ---------------------------------------------------------- CPU baseline

def cpu_baseline(wk, tokens, r):
    """The CPU oracle on the first `tokens` tokens of the same workload (all
    of them by default): the seven projections, then the per-head QK^T, each
    timed on its own."""
    import oracle.rmm_oracle as ro
    import workloads as wl
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:                                  # threadpoolctl missing
        blas_threads = os.cpu_count() or 1
    X = {n: wl.decode(wl.f32_to_bf16_bits(wl.workload_input(wk, n, M=tokens)), "bf16")
         for n in wk.inputs}
    W = {p.name: wl.decode(wl.f32_to_bf16_bits(wl.workload_weight(wk, p)), "bf16")
         for p in wk.projections}
    q, k = wl.workload_qk(wk, L=tokens)
    Q = wl.decode(wl.f32_to_bf16_bits(q), "bf16")
    Kc = wl.decode(wl.f32_to_bf16_bits(k), "bf16")
    del q, k
    a = wk.attention
    t0 = time.perf_counter()
    f_proj = 0
    for p in wk.projections:
        Y, idx, _ = ro.rmm(X[p.input_name], W[p.name], r)
        f_proj += 2 * tokens * p.N * len(idx)
        del Y
    t1 = time.perf_counter()
    S, qidx, _ = ro.rmm_qk(Q, Kc, r, True)
    f_qk = 2 * a.H * (tokens * (tokens + 1) // 2) * qidx.shape[1]
    del S
    t2 = time.perf_counter()
    dt = t2 - t0
    scope = "all" if tokens == wk.M else f"the first {tokens} of {wk.M}"
    return {"value": (f_proj + f_qk) / dt / 1e12, "unit": "TFLOP/s", "cores": int(blas_threads),
            "kind": "oracle",
            "projections": {"gflop": round(f_proj / 1e9, 1), "s": round(t1 - t0, 2),
                            "tflops": round(f_proj / (t1 - t0) / 1e12, 4)},
            "qk": {"gflop": round(f_qk / 1e9, 1), "s": round(t2 - t1, 2),
                   "tflops": round(f_qk / (t2 - t1) / 1e12, 4)},
            "sample": (f"{scope} tokens of the same layer (all 7 projections + per-head QK^T, "
                       f"r={r}); {(f_proj + f_qk) / 1e9:.1f} retained GFLOP in {dt:.1f} s; "
                       f"float64, BLAS threads={blas_threads}, host cpus={os.cpu_count()}")}


def child_processes():
    """Processes this run started that are still alive (none expected)."""
    try:
        import psutil
        return [f"{c.pid}:{c.name()}" for c in psutil.Process().children(recursive=True)]
    except Exception as e:                              # psutil missing
        return [f"unknown ({type(e).__name__})"]


# ------------------------------------------------------------------ main

def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the library has no "
              "multi-GPU path. Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2608_13426_amd  # noqa: F401  (fails loudly without librmm.so)
    import workloads as wl
    dev = torch.device("cuda:0")
    if args.workload not in wl.WORKLOADS:
        sys.exit(f"unknown workload {args.workload!r}; known: {', '.join(sorted(wl.WORKLOADS))}")
    wk = wl.WORKLOADS[args.workload]
    if wk.attention is None or wk.dtype != "bf16" or \
            {"attn_in", "o_in", "mlp_in", "down_in"} - set(wk.inputs):
        sys.exit(f"bench.py times a whole bf16 decoder layer (layer_8b, layer_70b); "
                 f"{args.workload!r} is a parity-test workload")
    ratios = [float(x) for x in args.ratios.split(",")]
    if HEADLINE_R not in ratios:
        ratios.append(HEADLINE_R)
    t_gen = time.perf_counter()
    L = Layer(wk, dev)
    if args.copy_probe_mib > 0:
        n = args.copy_probe_mib << 20
        a = torch.empty(n, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b
    torch.cuda.synchronize()
    print(f"# inputs resident in HBM ({time.perf_counter() - t_gen:.1f} s)", file=sys.stderr,
          flush=True)
    sweep = {}
    for r in ratios:
        sweep[r] = time_ratio(L, r, args.steps, args.warmup)
        print(f"# r={r}: {sweep[r]['ms_per_step']:.3f} ms/step, "
              f"{sweep[r]['tflops']:.1f} TFLOP/s, GEMM {sweep[r]['gemm_tflops']:.1f} TFLOP/s",
              file=sys.stderr, flush=True)
    head = sweep[HEADLINE_R]
    base = sweep.get(1.0)
    for r, rec in sweep.items():
        rec["speedup_vs_r1"] = (base["ms_per_step"] / rec["ms_per_step"]) if base else None
    # the GEMM over every timed launch of the run (all ratios)
    g_ms = sum(rec["gemm_ms_total"] for rec in sweep.values())
    g_gflop = sum(rec["gemm_gflop_total"] for rec in sweep.values())
    g_n = sum(rec["gemm_launches"] for rec in sweep.values())
    roof_ach = g_gflop / g_ms        # GFLOP/ms = TFLOP/s
    out = {
        "metric": METRIC,
        "value": round(head["tflops"], 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(head["ms_per_step"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{wk.name}: {wk.description}", "seq_len": wk.M, "batch": 1,
                   "r": HEADLINE_R, "projections": [p.name for p in wk.projections],
                   "attention": f"per-head reduced QK^T, causal, {wk.attention.H} q / "
                                f"{wk.attention.Hkv} kv heads, d={wk.attention.D}"},
        "speedup_vs_r1": round(head["speedup_vs_r1"], 3) if base else None,
        "sweep": {str(r): {k: (round(v, 4) if isinstance(v, float) else v)
                           for k, v in rec.items()} for r, rec in sweep.items()},
        "roofline": {"bound": "mfma", "kernel": GEMM_KERNEL,
                     "achieved": round(roof_ach, 2), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(roof_ach / PEAK_BF16_TFLOPS, 4),
                     "traffic": recorded_traffic(
                         GEMM_TRAFFIC, f"{wk.name} r={','.join(str(r) for r in sorted(sweep))} grouped"),
                     "traffic_unit": "HBM bytes per launch (FETCH_SIZE + WRITE_SIZE)",
                     "launches": g_n,
                     "avg_launch_us": round(g_ms * 1e3 / g_n, 2),
                     "avg_launch_gflop": round(g_gflop / g_n, 3),
                     "ratios": sorted(sweep)},
    }
    if not args.no_policies:
        pol = {}
        for name, policy in POLICIES.items():
            rec = time_ratio(L, policy, args.steps, args.warmup)
            rec["speedup_vs_r1"] = (base["ms_per_step"] / rec["ms_per_step"]) if base else None
            pol[name] = {k: (round(v, 4) if isinstance(v, float) else v) for k, v in rec.items()}
            print(f"# policy {name}: {rec['ms_per_step']:.3f} ms/step, {rec['tflops']:.1f} TFLOP/s",
                  file=sys.stderr, flush=True)
        out["component_ratios"] = {
            "op": "the same step with a retention ratio per component (attn_in: q|k|v, o_in: o, "
                  "mlp_in: gate|up, down_in: down, qk: per-head QK^T); speedup over the "
                  "same pipeline at r = 1",
            "policies": pol,
        }
    if not args.no_fused_attention:
        att = {r: time_attention(L, r, args.steps, args.warmup) for r in sorted(sweep)}
        sdpa_us = time_sdpa(L, args.steps, args.warmup)
        print(f"# torch SDPA (dense, causal): {sdpa_us} us/call", file=sys.stderr, flush=True)
        for r, rec in att.items():
            print(f"# fused attention r={r}: {rec['avg_call_us']:.1f} us/call, "
                  f"{rec['retained_tflops']:.1f} TFLOP/s", file=sys.stderr, flush=True)
        a_ms = sum(rec["avg_call_us"] * rec["calls"] for rec in att.values()) * 1e-3
        a_gf = sum(rec["gflop"] * rec["calls"] for rec in att.values())
        a_ach = a_gf / a_ms
        a_h, a_1 = att.get(HEADLINE_R), att.get(1.0)
        out["fused_attention"] = {
            "op": "softmax(reduced QK^T + causal mask) V per head, S never written; "
                  f"{wk.attention.H} q / {wk.attention.Hkv} kv heads, seq {wk.M}, "
                  f"d={wk.attention.D}, V dense",
            "kernels": ["attn_compact_k_kernel", "attn_fwd_kernel"],
            "per_ratio": {str(r): {k: (round(v, 3) if isinstance(v, float) else v)
                                   for k, v in rec.items()} for r, rec in att.items()},
            "speedup_vs_r1": round(a_1["avg_call_us"] / a_h["avg_call_us"], 3) if a_1 else None,
            "speedup_bound": round(2.0 / (1.0 + HEADLINE_R), 3),
            "torch_sdpa_us": (round(sdpa_us, 1) if sdpa_us else None),
            "roofline": {"bound": "mfma", "kernel": "attn_fwd_kernel (+ attn_compact_k_kernel)",
                         "achieved": round(a_ach, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                         "frac": round(a_ach / PEAK_BF16_TFLOPS, 4),
                         "traffic": recorded_traffic(
                             ATTN_TRAFFIC, f"{wk.name} r={','.join(str(r) for r in sorted(att))}"),
                         "traffic_unit": "HBM bytes per call (FETCH_SIZE + WRITE_SIZE, both kernels)"},
        }
    if not args.no_attention_chain:
        ch = {r: time_attention_chain(L, r, args.steps, args.warmup) for r in sorted(sweep)}
        for r, rec in ch.items():
            print(f"# attention -> o-projection r={r}: fused {rec['fused_us']:.1f} us, unfused "
                  f"{rec['unfused_us']:.1f} us ({rec['layout_copy_us']:.1f} us of it the layout "
                  f"copy)", file=sys.stderr, flush=True)
        out["attention_o_chain"] = {
            "op": "reduced attention block feeding the reduced output projection (o, 4096 x "
                  "4096): fused = the block writes the projection's K-major input and its "
                  "column energies (no scoring pass), unfused = block, token-major layout "
                  "copy, scoring pass with K-major copy; both then TopK and K-major GEMM",
            "kernels": ["attn_compact_k_kernel", "attn_fwd_kernel", "score_finalize_kernel",
                        "select_kernel", "gemm_kmajor_tr_kernel"],
            "per_ratio": {str(r): {k: (round(v, 3) if isinstance(v, float) else v)
                                   for k, v in rec.items()} for r, rec in ch.items()},
        }
    if not args.no_mlp_chain:
        mc = {r: time_mlp_chain(L, r, args.steps, args.warmup) for r in sorted(sweep)}
        for r, rec in mc.items():
            print(f"# MLP chain r={r}: fused {rec['fused_us']:.1f} us, unfused "
                  f"{rec['unfused_us']:.1f} us ({rec['activation_us']:.1f} us of it the torch "
                  f"activation)", file=sys.stderr, flush=True)
        out["mlp_chain"] = {
            "op": "the layer's MLP: gate|up (4096 -> 2 x 14336) then down (14336 -> 4096), "
                  "each reduced at r; fused = the gate|up GEMM's epilogue applies silu(g)*u "
                  "and writes the down projection's K-major input and its column energies "
                  "(no scoring pass over it), unfused = gate|up GEMM, torch activation, "
                  "scoring pass with K-major copy; both then TopK and the down GEMM",
            "kernels": ["score_tile_kernel", "select_kernel", "gemm_kmajor_tr_kernel",
                        "score_finalize_kernel"],
            "per_ratio": {str(r): {k: (round(v, 3) if isinstance(v, float) else v)
                                   for k, v in rec.items()} for r, rec in mc.items()},
        }
    if not args.no_norm_chain:
        nc = {}
        for name in ("attn_in", "mlp_in"):
            for r in sorted(sweep):
                rec = time_norm_chain(L, name, r, args.steps, args.warmup)
                nc[f"{name}@{r}"] = {k: (round(v, 3) if isinstance(v, float) else v)
                                     for k, v in rec.items()}
                print(f"# norm -> {name} projection r={r}: fused {rec['fused_us']:.1f} us, unfused "
                      f"{rec['unfused_us']:.1f} us (torch norm {rec['torch_norm_us']:.1f} us); "
                      f"producer {rec['producer_us']:.1f} us ({rec['producer_gbs']:.0f} GB/s), "
                      f"scoring pass {rec['score_kmajor_us']:.1f} us", file=sys.stderr, flush=True)
        p_us = sum(v["producer_us"] for v in nc.values())
        p_b = sum(v["producer_bytes"] for v in nc.values())
        out["norm_chain"] = {
            "op": "RMSNorm in front of a projection group feeding its reduced GEMM: fused = "
                  "rmm_rmsnorm_kmajor writes the normalised rows K-major with their column "
                  "energies in one pass over X (no scoring pass), unfused = torch RMSNorm, "
                  "rmm_score_kmajor; both then TopK and the K-major GEMM (q|k|v or gate|up)",
            "kernels": ["rms_block_kmajor_kernel", "score_finalize_grouped_kernel",
                        "select_kernel", "gemm_kmajor_tr_kernel"],
            "per_input_ratio": nc,
            "roofline": {"bound": "hbm", "kernel": "rmm_rmsnorm_kmajor (both kernels)",
                         "achieved": round(p_b / (p_us * 1e-6) / 1e9, 1), "peak": PEAK_HBM_GBS,
                         "unit": "GB/s", "frac": round(p_b / (p_us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4),
                         "bytes_basis": "one read of X + one write of Xt + the energies per call",
                         "traffic": recorded_traffic(
                             NORM_TRAFFIC, f"{wk.name} attn_in,mlp_in"),
                         "traffic_unit": "HBM bytes per call (FETCH_SIZE + WRITE_SIZE, both kernels)"},
        }
    if not args.no_decode:
        dec = {r: time_decode(L, r, args.steps, args.warmup) for r in sorted(sweep)}
        for r, rec in dec.items():
            print(f"# decode step r={r}: {rec['us_per_step_grouped_graph']:.1f} us grouped as a graph "
                  f"({rec['us_per_step_grouped_eager']:.1f} us eager; separate calls "
                  f"{rec['us_per_step_separate']:.1f} us as a graph), reduced products "
                  f"{rec['gemv_us_per_step']:.1f} us ({rec['gemv_gbs']:.0f} GB/s)",
                  file=sys.stderr, flush=True)
        d_us = sum(rec["gemv_us_per_step"] * args.steps for rec in dec.values())
        d_b = sum(rec["gemv_bytes_per_step"] * args.steps for rec in dec.values())
        d_ach = d_b / (d_us * 1e-6) / 1e9
        d_h, d_1 = dec.get(HEADLINE_R), dec.get(1.0)
        out["decode"] = {
            "op": "one decode step, batch 1: per projection group of the layer (q|k|v, o, "
                  "gate|up, down) TopK of the token's squared activations, reduced product "
                  "over the retained weight rows (the four groups taken as independent); "
                  "rmm_decode_step runs all groups in three launches (us_per_step: the faster "
                  "of its eager launches and its HIP-graph replay); us_per_step_separate "
                  "replays the per-group calls (three launches each) as a graph",
            "kernels": ["select_token16_grouped_kernel", "gemv_partial_grouped_kernel",
                        "gemv_reduce_grouped_kernel"],
            "per_ratio": {str(r): {k: (round(v, 3) if isinstance(v, float) else v)
                                   for k, v in rec.items()} for r, rec in dec.items()},
            "speedup_vs_r1": round(d_1["us_per_step"] / d_h["us_per_step"], 3) if d_1 else None,
            "roofline": {"bound": "hbm", "kernel": "gemv_partial_grouped_kernel (+ gemv_reduce_grouped_kernel)",
                         "achieved": round(d_ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                         "frac": round(d_ach / PEAK_HBM_GBS, 4),
                         "traffic": recorded_traffic(
                             DECODE_TRAFFIC, f"{wk.name} r={','.join(str(r) for r in sorted(dec))} B=1"),
                         "traffic_unit": "HBM bytes per products call (FETCH_SIZE + WRITE_SIZE, mean "
                                         "over the ratios)"},
        }
    if not args.no_decode_batched:
        recs = [time_decode_batched(L, r, B, args.steps, args.warmup)
                for B in (4, 16, 32) for r in (0.25, 0.5, 1.0)]
        for rec in recs:
            print(f"# decode products B={rec['batch']} r={rec['r']}: shared {rec['shared_us']:.1f} us "
                  f"({rec['shared_gbs']:.0f} GB/s), per sequence {rec['per_sequence_us']:.1f} us, "
                  f"dense torch {rec['dense_torch_us']:.1f} us", file=sys.stderr, flush=True)
        head = next(x for x in recs if x["batch"] == 16 and x["r"] == HEADLINE_R)
        out["decode_batched"] = {
            "op": "the products of one decode step for B sequences (q|k|v, o, gate|up, down; each "
                  "sequence its own TopK set): rmm_decode_products reads k rows per sequence, "
                  "rmm_decode_products_shared reads each row of the union of the B sets once and "
                  "multiplies all sequences on the matrix cores; torch's dense product of the same "
                  "tokens; each a replayed graph of 10 back-to-back calls",
            "kernels": ["share_offsets_kernel", "share_union_kernel",
                        "share_product_kernel<128, 6> (B < 8), <256, 4> (B >= 8)", "share_reduce_kernel"],
            "per_batch_ratio": {f"B{x['batch']}@{x['r']}": {k: (round(v, 3) if isinstance(v, float) else v)
                                                           for k, v in x.items()} for x in recs},
            "roofline": {"bound": "hbm", "kernel": "rmm_decode_products_shared (all four kernels), B=16 "
                                                   f"r={HEADLINE_R}",
                         "achieved": round(head["shared_gbs"], 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                         "frac": round(head["shared_gbs"] / PEAK_HBM_GBS, 4),
                         "bytes_basis": "the union rows of every W once + the tokens and outputs",
                         "traffic": recorded_traffic(SHARED_TRAFFIC, f"{wk.name} B=16 r={HEADLINE_R}"),
                         "traffic_unit": "HBM bytes per call (FETCH_SIZE + WRITE_SIZE, all four kernels)"},
        }
    if not (args.no_pv_chain and args.no_pv):
        # the value-product records take the layer's causal scores at the
        # headline ratio (one untimed step leaves them in L.S, with the
        # per-head selection in L.qidx), whatever ran before
        run_step(L, HEADLINE_R)
    if not args.no_pv_chain:
        import torch
        import paper_2608_13426_amd as rmm
        a = wk.attention
        bufs = {"Pt": torch.empty((1, a.H, a.L, a.L), dtype=torch.bfloat16, device=L.dev),
                "e": torch.empty(a.H * a.L, dtype=torch.float64, device=L.dev),
                "ws": torch.empty(rmm.rmm_attention_weights_kmajor_workspace_size(1, a.H, a.L, a.L),
                                  dtype=torch.uint8, device=L.dev),
                "P": torch.empty((a.H, a.L, a.L), dtype=torch.bfloat16, device=L.dev),
                "Vr": L.V[0].repeat_interleave(a.H // a.Hkv, dim=0).contiguous(),
                "Od": torch.empty((a.H, a.L, a.D), dtype=torch.bfloat16, device=L.dev),
                "rmax": torch.empty(a.H * a.L, dtype=torch.float32, device=L.dev),
                "rinv": torch.empty(a.H * a.L, dtype=torch.float32, device=L.dev)}
        pc = {r: time_pv_chain(L, r, args.steps, args.warmup, bufs) for r in sorted(sweep)}
        del bufs
        torch.cuda.empty_cache()
        for r, rec in pc.items():
            print(f"# PV chain r={r}: reduced {rec['reduced_us']:.1f} us (producer "
                  f"{rec['producer_us']:.1f} us at {rec['producer_gbs']:.0f} GB/s, product "
                  f"{rec['product_us']:.1f} us); dense torch softmax + P@V {rec['dense_torch_us']:.1f} us; "
                  f"from QK: {rec['from_qk_us']:.1f} us, with QK row statistics "
                  f"{rec['from_qk_rowstats_us']:.1f} us (QK {rec['qk_us']:.1f} -> "
                  f"{rec['qk_rowstats_us']:.1f} us, producer {rec['producer_rowstats_us']:.1f} us at "
                  f"{rec['producer_rowstats_gbs']:.0f} GB/s)", file=sys.stderr, flush=True)
        c_h, c_1 = pc.get(HEADLINE_R), pc.get(1.0)
        p_us = sum(v["producer_us"] for v in pc.values())
        p_b = sum(v["producer_bytes"] for v in pc.values())
        out["pv_chain"] = {
            "op": "scores -> attention weights -> token-axis reduced value product per query head: "
                  "reduced = rmm_attention_weights_kmajor (weights K-major + token energies, the "
                  "causally masked half of S not read), TopK per head, rmm_reduced_pv_kmajor (kept "
                  "token rows, causal row tiles trimmed); dense = torch softmax + torch P @ V; "
                  f"{a.H} q / {a.Hkv} kv heads, seq {wk.M}, d={a.D}",
            "kernels": ["softmax_rowstats_kernel", "score_tile_kernel (softmax variant)",
                        "score_finalize_kernel", "select_kernel", "gemm_kmajor_tr_kernel (256x128)"],
            "per_ratio": {str(r): {k: (round(v, 3) if isinstance(v, float) else v)
                                   for k, v in rec.items()} for r, rec in pc.items()},
            "speedup_vs_r1": round(c_1["reduced_us"] / c_h["reduced_us"], 3) if c_1 and c_h else None,
            "speedup_vs_dense_torch": round(c_h["speedup_vs_dense_torch"], 3) if c_h else None,
            "roofline": {"bound": "hbm", "kernel": "rmm_attention_weights_kmajor (all three kernels)",
                         "achieved": round(p_b / (p_us * 1e-6) / 1e9, 1), "peak": PEAK_HBM_GBS,
                         "unit": "GB/s", "frac": round(p_b / (p_us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4),
                         "bytes_basis": "the causal part of S read once + the stored part of Pt + "
                                        "energies per call (the implementation reads S twice: row "
                                        "statistics, then the weights)",
                         "traffic": None},
            "rowstats_speedup_from_qk": round(c_h["rowstats_speedup"], 3) if c_h else None,
            "roofline_rowstats": {
                "bound": "hbm",
                "kernel": "rmm_attention_weights_kmajor_rowstats (score_tile_kernel softmax variant "
                          "+ score_finalize_kernel; row statistics from rmm_reduced_qk_rowstats)",
                "achieved": round(c_h["producer_rowstats_gbs"], 1) if c_h else None,
                "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(c_h["producer_rowstats_gbs"] / PEAK_HBM_GBS, 4) if c_h else None,
                "bytes_basis": "as roofline (S read once by this pass)", "traffic": None},
        }
    if not args.no_pv:
        import torch
        import paper_2608_13426_amd as rmm
        a = wk.attention
        attention_weights(L)
        ws = torch.empty(rmm.rmm_workspace_size(rmm.RMM_OP_PV, a.H, a.L, a.L, a.L),
                         dtype=torch.uint8, device=L.dev)
        pv = {r: time_pv(L, r, args.steps, args.warmup, ws) for r in sorted(sweep)}
        del ws
        dense_us = time_dense_pv(L, args.steps, args.warmup)
        for r, rec in pv.items():
            print(f"# token-axis PV r={r}: {rec['avg_call_us']:.1f} us/call "
                  f"({rec['gbs']:.0f} GB/s of one P read); dense P@V {dense_us:.1f} us",
                  file=sys.stderr, flush=True)
        p_us = sum(rec["avg_call_us"] * rec["calls"] for rec in pv.values())
        p_b = sum(rec["bytes"] * rec["calls"] for rec in pv.values())
        p_ach = p_b / (p_us * 1e-6) / 1e9
        p_h, p_1 = pv.get(HEADLINE_R), pv.get(1.0)
        out["pv_token"] = {
            "op": "token-axis reduced value product per query head: TopK of the column norms "
                  "of the attention weights P (softmax of the layer's causal scores), then "
                  f"P[:, T] V[T, :]; {wk.attention.H} q / {wk.attention.Hkv} kv heads, "
                  f"seq {wk.M}, d={wk.attention.D}",
            "kernels": ["score_tile_kernel", "score_finalize_kernel", "select_kernel",
                        "gemm_kmajor_tr_kernel"],
            "per_ratio": {str(r): {k: (round(v, 3) if isinstance(v, float) else v)
                                   for k, v in rec.items()} for r, rec in pv.items()},
            "speedup_vs_r1": round(p_1["avg_call_us"] / p_h["avg_call_us"], 3) if p_1 else None,
            "dense_torch_us": round(dense_us, 1),
            "speedup_vs_dense_torch": round(dense_us / p_h["avg_call_us"], 3) if p_h else None,
            "roofline": {"bound": "hbm", "kernel": "rmm_reduced_pv (all kernels of a call)",
                         "achieved": round(p_ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                         "frac": round(p_ach / PEAK_HBM_GBS, 4), "traffic": None,
                         "bytes_basis": "one read of P + kept V rows + O per call"},
        }
    if not args.no_layer_forward:
        lf = time_layer_forward(L, args.steps, args.warmup)
        print(f"# layer forward: rmm " + ", ".join(f"r={r} {lf[f'rmm_ms@{r}']:.3f} ms"
                                                   for r in (0.5, 0.8, 1.0))
              + f"; torch dense {lf.get('torch_dense_ms')} ms", file=sys.stderr, flush=True)
        out["layer_forward"] = {
            "op": "one prefill pass of the whole decoder layer (batch 1, seq "
                  f"{wk.M}, no rotary embedding): RMSNorm producers, reduced q|k|v, per-head "
                  "reduced attention writing the o-projection's K-major input, reduced o, "
                  "residual, RMSNorm producer, reduced gate|up with the SwiGLU producer, reduced "
                  "down, residual; every product at ratio r; against torch's dense layer "
                  "(fp32 RMSNorm, x @ W, fused SDPA, silu(g) * u)",
            "per_ratio": lf,
        }
    if not args.no_paper_kernels:
        pk = time_paper_kernels(wk, L.dev, args.steps, args.warmup)
        for Ln, rec in pk.items():
            print(f"# paper kernels L={Ln}: QK^T rmm {rec['qk_rmm_us@0.8']:.1f} us (r=1 "
                  f"{rec['qk_rmm_us@1.0']:.1f}, dense torch {rec['qk_dense_torch_us']:.1f}); "
                  f"AV rmm {rec['av_rmm_us@0.8']:.1f} us (r=1 {rec['av_rmm_us@1.0']:.1f}, dense "
                  f"torch {rec['av_dense_torch_us']:.1f}); AV from S rmm {rec['av_chain_rmm_us@0.8']:.1f} "
                  f"us (r=1 {rec['av_chain_rmm_us@1.0']:.1f}, dense torch softmax + P@V "
                  f"{rec['av_chain_dense_torch_us']:.1f})", file=sys.stderr, flush=True)
        out["paper_kernels"] = {
            "op": "the paper's kernel-level latency benchmark (Sec. 6): per sequence length, "
                  "reduced QK^T (per-head scoring + TopK + rmm_reduced_qk writing the masked S) "
                  "and reduced AV (rmm_reduced_pv on row-major P: column norms + TopK + gathered "
                  "product; av_chain: from the scores, the weights written K-major with their "
                  "token energies + TopK + product) at rho = 0.8 and 1, against torch's dense bf16 "
                  "products (av_chain: torch softmax + P @ V); "
                  f"{wk.attention.H} q / {wk.attention.Hkv} kv heads, d={wk.attention.D}, causal, "
                  "batch 1; paper_a100_ms: the paper's own dense and RMM times on an A100 "
                  "(context, other hardware)",
            "rho": 0.8,
            "per_length": {str(Ln): rec for Ln, rec in pk.items()},
        }
    if not args.no_cpu_baseline:
        tokens = args.cpu_tokens or wk.M
        print(f"# CPU oracle on {tokens} tokens ...", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(wk, tokens, HEADLINE_R)
    out["children_at_exit"] = child_processes()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
