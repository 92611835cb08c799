"""C-ABI checks that need no GPU: the library loads, exports every symbol the
header declares, and its host-side logic (k rule, workspace sizes, argument
validation) behaves as documented.  Only calls that fail validation are made
here; validation happens before any HIP call."""
import ctypes
import math
import os
import re
from fractions import Fraction

import pytest

import paper_2608_13426_amd as rmm
from oracle import rmm_oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rmm.h")

OK, INVALID, UNSUPPORTED, WS_SMALL, HIP, TOO_LARGE = 0, 1, 2, 3, 4, 5
P = ctypes.c_void_p(0x100000)          # a non-null pointer that is never dereferenced
NULL = None


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rmm_[a-z_]+)\s*\(", text)))


def test_header_symbols_are_exported():
    names = _declared()
    assert names == sorted(rmm.EXPORTED_SYMBOLS)
    for n in names:
        assert hasattr(rmm.lib, n), n


def test_library_is_gfx950_code_object():
    data = open(rmm.LIB_PATH, "rb").read()
    assert b"gfx950" in data


def test_retained_count_matches_rule():
    for K in (1, 2, 7, 100, 128, 512, 4096, 14336, 28672):
        for p in range(1, 101):
            s = f"{p / 100:.2f}"
            want = max(1, math.ceil(Fraction(s) * K))
            assert rmm.rmm_retained_count(float(s), K) == want
            assert rmm.rmm_retained_count(float(s), K) == rmm_oracle.retained_count(float(s), K)
    assert rmm.rmm_retained_count(0.07, 100) == 7
    assert rmm.rmm_retained_count(0.8, 128) == 103
    for bad in (0.0, -1.0, 1.0000001, float("nan"), float("inf")):
        assert rmm.rmm_retained_count(bad, 128) == -1
    assert rmm.rmm_retained_count(0.5, 0) == -1
    assert rmm.rmm_retained_count(0.5, 2 ** 31) == -1


def test_workspace_sizes():
    # score: one float64 partial per (unit, split, column); none when unsplit
    ws = rmm.rmm_workspace_size(rmm.RMM_OP_SCORE, 1, 8192, 4096)
    assert ws > 0 and ws % 8 == 0
    assert rmm.rmm_workspace_size(rmm.RMM_OP_SCORE, 1, 32, 512) == 0
    assert rmm.rmm_workspace_size(rmm.RMM_OP_SELECT, 4, 100, 4096, 10) == 0
    lin = rmm.rmm_workspace_size(rmm.RMM_OP_LINEAR, 1, 8192, 4096, 2048)
    assert lin >= ws + 4096 * 8 + 2048 * 4
    assert rmm.rmm_workspace_size(rmm.RMM_OP_LINEAR, 1, 8192, 4096, 0) == 0
    assert rmm.rmm_workspace_size(rmm.RMM_OP_SCORE, 0, 8192, 4096) == 0


def test_status_strings():
    for code in range(6):
        s = rmm.rmm_status_string(code)
        assert isinstance(s, str) and s
    assert rmm.rmm_status_string(99) == "unknown status"


def test_score_validation():
    f = rmm.lib.rmm_score
    assert f(NULL, 1, 1, 8, 8, 8, P, NULL, 0, NULL) == INVALID
    assert f(P, 1, 1, 8, 8, 8, NULL, NULL, 0, NULL) == INVALID
    assert f(P, 7, 1, 8, 8, 8, P, NULL, 0, NULL) == INVALID        # dtype
    assert f(P, 1, 0, 8, 8, 8, P, NULL, 0, NULL) == INVALID        # B
    assert f(P, 1, 1, 0, 8, 8, P, NULL, 0, NULL) == INVALID        # M
    assert f(P, 1, 1, 8, 0, 8, P, NULL, 0, NULL) == INVALID        # K
    assert f(P, 1, 1, 8, 8, 7, P, NULL, 0, NULL) == INVALID        # ldx < K
    assert f(P, 1, 70000, 8, 8, 8, P, NULL, 0, NULL) == UNSUPPORTED
    need = rmm.rmm_workspace_size(rmm.RMM_OP_SCORE, 1, 8192, 4096)
    assert f(P, 1, 1, 8192, 4096, 4096, P, NULL, 0, NULL) == WS_SMALL
    assert f(P, 1, 1, 8192, 4096, 4096, P, P, need - 8, NULL) == WS_SMALL
    assert f(P, 1, 1, 8192, 4096, 4096, P, ctypes.c_void_p(0x100004), need, NULL) == INVALID


def test_score_kmajor_validation():
    f = rmm.lib.rmm_score_kmajor
    A = ctypes.c_void_p(0x100000)       # 16-byte aligned, never dereferenced
    assert f(A, 1, 64, 128, 128, P, NULL, 64, NULL, 0, NULL) == INVALID        # no Xt
    assert f(A, 1, 64, 128, 128, P, A, 60, NULL, 0, NULL) == INVALID          # ldxt < M
    assert f(A, 1, 64, 130, 130, P, A, 64, NULL, 0, NULL) == UNSUPPORTED      # ldx % 8
    assert f(A, 1, 64, 128, 128, P, A, 68, NULL, 0, NULL) == UNSUPPORTED      # ldxt % 8
    assert f(ctypes.c_void_p(0x100002), 1, 64, 128, 128, P, A, 64, NULL, 0, NULL) == UNSUPPORTED
    assert f(NULL, 1, 64, 128, 128, P, A, 64, NULL, 0, NULL) == INVALID


def test_gemm_kmajor_validation():
    f = rmm.lib.rmm_reduced_gemm_kmajor
    A = ctypes.c_void_p(0x100000)
    ok = [A, A, P, 1, 64, 64, 128, 32, 64, 64, A, 64, NULL]

    def call(i, v):
        a = list(ok)
        a[i] = v
        return f(*a)

    for i in (0, 1, 2, 10):
        assert call(i, NULL) == INVALID
    assert call(7, 0) == INVALID            # k
    assert call(7, 129) == INVALID          # k > K
    assert call(8, 63) == INVALID           # ldxt < M
    assert call(8, 68) == UNSUPPORTED       # ldxt % 8
    assert call(9, 60) == INVALID           # ldw < N
    assert call(0, ctypes.c_void_p(0x100008)) == UNSUPPORTED
    assert call(6, 2 ** 24) == UNSUPPORTED  # K * ldxt * 2 bytes beyond 2^31


def test_select_validation():
    f = rmm.lib.rmm_select
    assert f(NULL, 1, 8, 2, P, NULL) == INVALID
    assert f(P, 1, 8, 2, NULL, NULL) == INVALID
    assert f(P, 0, 8, 2, P, NULL) == INVALID
    assert f(P, 1, 8, 0, P, NULL) == INVALID
    assert f(P, 1, 8, 9, P, NULL) == INVALID
    assert f(P, 1, 0, 1, P, NULL) == INVALID
    assert f(P, 1, 2 ** 31, 1, P, NULL) == INVALID


def test_gemm_validation():
    f = rmm.lib.rmm_reduced_gemm
    args = dict(X=P, W=P, idx=P, dt=1, B=1, M=16, N=16, K=32, k=8, ldx=32, ldw=16, Y=P, ldy=16)

    def call(**kw):
        a = {**args, **kw}
        return f(a["X"], a["W"], a["idx"], a["dt"], a["B"], a["M"], a["N"], a["K"], a["k"],
                 a["ldx"], a["ldw"], a["Y"], a["ldy"], NULL)

    for name in ("X", "W", "idx", "Y"):
        assert call(**{name: NULL}) == INVALID, name
    assert call(dt=5) == INVALID
    for name in ("B", "M", "N", "K"):
        assert call(**{name: 0}) == INVALID, name
    assert call(k=0) == INVALID
    assert call(k=33) == INVALID
    assert call(ldx=31) == INVALID
    assert call(ldw=15) == INVALID
    assert call(ldy=15) == INVALID
    assert call(B=70000) == UNSUPPORTED


def test_qk_validation():
    f = rmm.lib.rmm_reduced_qk
    base = [P, P, P, 1, 1, 32, 8, 64, 64, 128, 64, ctypes.c_float(0.088), 1, P, NULL]

    def call(i, v):
        a = list(base)
        a[i] = v
        return f(*a)

    for i in (0, 1, 2, 13):
        assert call(i, NULL) == INVALID
    assert call(3, 9) == INVALID           # dtype
    assert call(4, 0) == INVALID           # batch
    assert call(6, 5) == INVALID           # H % Hkv
    assert call(10, 0) == INVALID          # k
    assert call(10, 129) == INVALID        # k > D
    assert call(9, 512) == UNSUPPORTED     # D > 256


def test_attention_validation():
    f = rmm.lib.rmm_reduced_attention
    A = ctypes.c_void_p(0x100000)
    need = rmm.rmm_workspace_size(rmm.RMM_OP_ATTENTION, 8, 64, 128, 64)
    base = [A, A, A, P, 1, 1, 8, 2, 64, 64, 128, 64, ctypes.c_float(0.088), 1, A, A, need, NULL]

    def call(i, v):
        a = list(base)
        a[i] = v
        return f(*a)

    for i in (0, 1, 2, 3, 14):
        assert call(i, NULL) == INVALID
    assert call(4, 9) == INVALID            # dtype
    assert call(5, 0) == INVALID            # batch
    assert call(7, 3) == INVALID            # H % Hkv
    assert call(11, 0) == INVALID           # k
    assert call(11, 129) == INVALID         # k > D
    assert call(4, 0) == UNSUPPORTED        # fp32
    assert call(10, 64) == UNSUPPORTED      # D != 128
    assert call(2, ctypes.c_void_p(0x100008)) == UNSUPPORTED   # V not 16-byte aligned
    assert call(15, NULL) == WS_SMALL       # no workspace
    assert call(16, need - 1) == WS_SMALL
    assert call(15, ctypes.c_void_p(0x100008)) == INVALID      # workspace not 16-byte aligned


def test_attention_workspace_size():
    # each query head's retained key dims as rows of kp = 32, 64, 96 or 128 bf16
    for k, kp in ((1, 32), (32, 32), (33, 64), (64, 64), (65, 96), (96, 96), (97, 128), (128, 128)):
        assert rmm.rmm_workspace_size(rmm.RMM_OP_ATTENTION, 32, 8192, 128, k) == 32 * 8192 * kp * 2
    assert rmm.rmm_workspace_size(rmm.RMM_OP_ATTENTION, 3, 70, 128, 5) == 3 * 70 * 32 * 2 // 256 * 256 + 256
    assert rmm.rmm_workspace_size(rmm.RMM_OP_ATTENTION, 1, 64, 128, 0) == 0
    assert rmm.rmm_workspace_size(rmm.RMM_OP_ATTENTION, 1, 64, 128, 129) == 0


def test_attention_kmajor_validation():
    f = rmm.lib.rmm_reduced_attention_kmajor
    A = ctypes.c_void_p(0x100000)
    need = rmm.rmm_attention_kmajor_workspace_size(1, 8, 64, 64, 128, 64)
    # Q Kc V idx dtype batch H Hkv Lq Lk D k scale causal Ot ldot energy ws ws_bytes stream
    base = [A, A, A, P, 1, 1, 8, 2, 64, 64, 128, 64, ctypes.c_float(0.088), 1, A, 64, A, A, need,
            NULL]

    def call(i, v):
        a = list(base)
        a[i] = v
        return f(*a)

    for i in (0, 1, 2, 3, 14, 16):
        assert call(i, NULL) == INVALID
    assert call(4, 9) == INVALID            # dtype
    assert call(5, 0) == INVALID            # batch
    assert call(7, 3) == INVALID            # H % Hkv
    assert call(11, 0) == INVALID           # k
    assert call(11, 129) == INVALID         # k > D
    assert call(15, 56) == INVALID          # ldot < Lq
    assert call(4, 0) == UNSUPPORTED        # fp32
    assert call(10, 64) == UNSUPPORTED      # D != 128
    assert call(14, ctypes.c_void_p(0x100008)) == UNSUPPORTED  # Ot not 16-byte aligned
    assert call(15, 68) == UNSUPPORTED      # ldot % 8
    assert call(16, ctypes.c_void_p(0x100004)) == UNSUPPORTED  # energy not 8-byte aligned
    a = list(base)
    a[8], a[15] = 60, 64                    # Lq % 8
    assert f(*a) == UNSUPPORTED
    assert call(17, NULL) == WS_SMALL       # no workspace
    assert call(18, need - 1) == WS_SMALL
    assert call(17, ctypes.c_void_p(0x100010)) == INVALID      # workspace not 256-byte aligned


def test_attention_kmajor_workspace_size():
    # compacted key rows (as rmm_reduced_attention), then one float64 partial
    # energy per (sequence, 256-query tile, output channel)
    n = rmm.rmm_attention_kmajor_workspace_size(1, 32, 8192, 8192, 128, 64)
    assert n == 32 * 8192 * 64 * 2 + 32 * 32 * 128 * 8
    n = rmm.rmm_attention_kmajor_workspace_size(2, 4, 300, 520, 128, 33)
    ki = 2 * 4 * 520 * 64 * 2
    assert n == (ki + 255) // 256 * 256 + (2 * 2 * 4 * 128 * 8 + 255) // 256 * 256
    assert rmm.rmm_attention_kmajor_workspace_size(1, 4, 64, 64, 128, 0) == 0
    assert rmm.rmm_attention_kmajor_workspace_size(1, 4, 0, 64, 128, 8) == 0


def test_gemm_swiglu_validation():
    f = rmm.lib.rmm_reduced_gemm_swiglu_kmajor
    A = ctypes.c_void_p(0x100000)
    need = rmm.rmm_gemm_swiglu_workspace_size(1, 512, 256)
    # Xt Wgu idx B M F K k ldxt ldw Ht ldht energy ws ws_bytes stream
    base = [A, A, P, 1, 512, 256, 300, 150, 512, 512, A, 512, A, A, need, NULL]

    def call(i, v):
        a = list(base)
        a[i] = v
        return f(*a)

    for i in (0, 1, 2, 10, 12):
        assert call(i, NULL) == INVALID
    assert call(3, 0) == INVALID            # B
    assert call(5, 0) == INVALID            # F
    assert call(7, 0) == INVALID            # k
    assert call(7, 301) == INVALID          # k > K
    assert call(8, 504) == INVALID          # ldxt < M
    assert call(9, 504) == INVALID          # ldw < 2F
    assert call(11, 504) == INVALID         # ldht < M
    assert call(5, 192) == UNSUPPORTED      # F % 128 (ldw 512 still >= 2F)
    a = list(base)
    a[4], a[8], a[11] = 500, 504, 504       # M % 8
    assert f(*a) == UNSUPPORTED
    assert call(11, 516) == UNSUPPORTED     # ldht % 8
    assert call(10, ctypes.c_void_p(0x100008)) == UNSUPPORTED  # Ht not 16-byte aligned
    assert call(1, ctypes.c_void_p(0x100008)) == UNSUPPORTED   # Wgu not 16-byte aligned
    assert call(12, ctypes.c_void_p(0x100004)) == UNSUPPORTED  # energy not 8-byte aligned
    assert call(13, NULL) == WS_SMALL
    assert call(14, need - 1) == WS_SMALL
    assert call(13, ctypes.c_void_p(0x100004)) == INVALID      # workspace not 8-byte aligned


def test_gemm_swiglu_workspace_size():
    # one float64 partial energy per (unit, 256-row tile, channel)
    assert rmm.rmm_gemm_swiglu_workspace_size(1, 8192, 14336) == 32 * 14336 * 8
    assert rmm.rmm_gemm_swiglu_workspace_size(2, 264, 128) == 2 * 2 * 128 * 8
    assert rmm.rmm_gemm_swiglu_workspace_size(1, 8, 128) == 1024
    assert rmm.rmm_gemm_swiglu_workspace_size(0, 8, 128) == 0


def test_check_indices_validation():
    f = rmm.lib.rmm_check_indices
    base = [P, 2, 8, 16, P, NULL]

    def call(i, v):
        a = list(base)
        a[i] = v
        return f(*a)

    assert call(0, NULL) == INVALID
    assert call(4, NULL) == INVALID
    for i, v in ((1, 0), (2, 0), (3, 0), (2, 17), (3, 2 ** 31)):
        assert call(i, v) == INVALID
    assert call(1, 2 ** 31) == UNSUPPORTED


def test_linear_validation():
    f = rmm.lib.rmm_linear
    need = rmm.rmm_workspace_size(rmm.RMM_OP_LINEAR, 1, 64, 128, 64)
    base = [P, P, 0.5, 1, 1, 64, 32, 128, 128, 32, P, 32, NULL, P, need, NULL]

    def call(i, v):
        a = list(base)
        a[i] = v
        return f(*a)

    assert call(2, 0.0) == INVALID
    assert call(2, 1.5) == INVALID
    assert call(2, float("nan")) == INVALID
    assert call(0, NULL) == INVALID
    assert call(13, NULL) == WS_SMALL
    assert call(14, need - 1) == WS_SMALL
    assert call(8, 100) == INVALID           # ldx < K


def test_binding_rejects_host_tensors():
    import torch
    x = torch.zeros(4, 8, dtype=torch.bfloat16)
    e = torch.zeros(8, dtype=torch.float64)
    with pytest.raises(ValueError):
        rmm.rmm_score(x, e)


def test_gemv_validation():
    f = rmm.lib.rmm_reduced_gemv
    need = rmm.rmm_gemv_workspace_size(1, 1, 4096, 2048)
    assert need > 0                          # one token: the list is split over slices
    base = [P, P, P, 1, 1, 1, 4096, 4096, 2048, 4096, 4096, P, 4096, P, need, NULL]

    def call(i, v):
        a = list(base)
        a[i] = v
        return f(*a)

    for i in (0, 1, 2, 11):
        assert call(i, NULL) == INVALID
    assert call(3, 7) == INVALID            # dtype
    assert call(3, 0) == UNSUPPORTED        # fp32
    assert call(5, 9) == UNSUPPORTED        # more than 8 rows per unit
    assert call(8, 0) == INVALID            # k
    assert call(10, 4000) == INVALID        # ldw < N
    assert call(13, NULL) == WS_SMALL
    assert call(14, need - 1) == WS_SMALL
    assert call(13, ctypes.c_void_p(0x100008)) == INVALID     # workspace not 16-byte aligned
    big = list(base)
    big[7], big[9], big[10] = 65536, 65536, 65536     # K * ldw * 2 reaches 2^33
    big[6], big[12] = 65536, 65536
    assert f(*big) == UNSUPPORTED


def test_pv_validation():
    f = rmm.lib.rmm_reduced_pv
    # P [1][4][64][96], V [1][2][96][128], kt = 48
    need = rmm.rmm_workspace_size(rmm.RMM_OP_PV, 4, 64, 96, 48)
    assert need == rmm.rmm_workspace_size(rmm.RMM_OP_LINEAR, 4, 64, 96, 48) > 0
    base = [P, P, 1, 1, 4, 2, 64, 96, 128, 96, 48, P, NULL, P, need, NULL]

    def call(i, v):
        a = list(base)
        a[i] = v
        return f(*a)

    for i in (0, 1, 11):
        assert call(i, NULL) == INVALID
    assert call(2, 7) == INVALID            # dtype
    assert call(5, 3) == INVALID            # H % Hkv != 0
    assert call(4, 0) == INVALID            # H
    assert call(10, 0) == INVALID           # kt < 1
    assert call(10, 97) == INVALID          # kt > Lk
    assert call(9, 95) == INVALID           # ldp < Lk
    assert call(13, NULL) == WS_SMALL
    assert call(14, need - 1) == WS_SMALL
    assert call(13, ctypes.c_void_p(0x100004)) == INVALID     # workspace not 8-byte aligned


def test_gemv_workspace_size():
    # many units and wide rows: one slice per workgroup column, no partials
    assert rmm.rmm_gemv_workspace_size(16, 1, 28672, 64) == 0
    # one unit: fp32 partials of every slice, 256-byte aligned
    n = rmm.rmm_gemv_workspace_size(1, 1, 4096, 2048)
    assert n > 0 and n % 256 == 0 and n % (4096 * 4) == 0
    assert rmm.rmm_gemv_workspace_size(1, 2, 4096, 2048) == 2 * n
    for bad in ((0, 1, 8, 8), (1, 0, 8, 8), (1, 9, 8, 8), (1, 1, 0, 8), (1, 1, 8, 0)):
        assert rmm.rmm_gemv_workspace_size(*bad) == 0


def test_select_tokens_validation():
    f = rmm.lib.rmm_select_tokens
    base = [P, 1, 2, 4096, 4096, 100, P, NULL]

    def call(i, v):
        a = list(base)
        a[i] = v
        return f(*a)

    assert call(0, NULL) == INVALID
    assert call(6, NULL) == INVALID
    assert call(1, 5) == INVALID            # dtype
    assert call(2, 0) == INVALID            # B
    assert call(3, 0) == INVALID            # K
    assert call(5, 0) == INVALID            # k
    assert call(5, 4097) == INVALID         # k > K
    assert call(4, 4095) == INVALID         # ldx < K


def test_linear_noalloc_validation():
    """Argument errors and the scratch limit are reported before any HIP call
    (this container has no GPU: a call that reached the device would fail
    with HIP instead)."""
    f = rmm.lib.rmm_linear_noalloc
    assert rmm.rmm_noalloc_scratch_bytes() == 64 << 20
    base = [P, P, 0.5, 1, 1, 64, 32, 128, 128, 32, P, 32, NULL, NULL]

    def call(i, v):
        a = list(base)
        a[i] = v
        return f(*a)

    assert call(2, 0.0) == INVALID
    assert call(2, float("nan")) == INVALID
    assert call(0, NULL) == INVALID
    assert call(1, NULL) == INVALID
    assert call(10, NULL) == INVALID
    assert call(3, 7) == INVALID             # dtype
    assert call(8, 100) == INVALID           # ldx < K
    # 8192 x 4096 bf16 activations: the K-major copy alone is 64 MiB
    big = [P, P, 0.5, 1, 1, 8192, 4096, 4096, 4096, 4096, P, 4096, NULL, NULL]
    assert rmm.rmm_workspace_size(rmm.RMM_OP_LINEAR, 1, 8192, 4096, 2048) > (64 << 20)
    assert f(*big) == TOO_LARGE
    assert rmm.rmm_status_string(TOO_LARGE) == "problem exceeds the library's fixed scratch buffer"


def test_rmsnorm_kmajor_validation():
    f = rmm.lib.rmm_rmsnorm_kmajor
    need = rmm.rmm_rmsnorm_kmajor_workspace_size(1, 64, 128)
    assert need > 0 and need % 8 == 0
    base = [P, P, 1e-5, 1, 64, 128, 128, P, 64, P, P, need, NULL]

    def call(i, v):
        a = list(base)
        a[i] = v
        return f(*a)

    for i in (0, 1, 7, 9):
        assert call(i, NULL) == INVALID
    assert call(2, -1.0) == INVALID
    assert call(2, float("nan")) == INVALID
    assert call(2, float("inf")) == INVALID
    assert call(3, 0) == INVALID
    assert call(6, 100) == INVALID            # ldx < K
    assert call(8, 63) == INVALID             # ldxt < M
    def call2(K, ldx):
        a = list(base)
        a[5], a[6] = K, ldx
        return f(*a)

    assert call2(130, 136) == UNSUPPORTED     # K % 8
    assert call(6, 132) == UNSUPPORTED        # ldx % 8
    assert call(0, ctypes.c_void_p(0x100008)) == UNSUPPORTED   # misaligned X
    assert call(10, NULL) == WS_SMALL
    assert call(11, need - 1) == WS_SMALL
    assert call(10, ctypes.c_void_p(0x100008)) == INVALID     # workspace not 256-byte aligned


def test_attention_weights_kmajor_validation():
    f = rmm.lib.rmm_attention_weights_kmajor
    need = rmm.rmm_attention_weights_kmajor_workspace_size(1, 2, 64, 96)
    assert need > 0 and need % 256 == 0
    base = [P, 1, 2, 64, 96, 96, 1, P, 64, P, P, need, NULL]

    def call(i, v):
        a = list(base)
        a[i] = v
        return f(*a)

    for i in (0, 7, 9):
        assert call(i, NULL) == INVALID
    assert call(5, 90) == INVALID             # lds < Lk
    assert call(8, 60) == INVALID             # ldpt < Lq
    assert call(5, 100) == UNSUPPORTED        # lds % 8
    assert call(10, NULL) == WS_SMALL
    assert call(11, need - 1) == WS_SMALL
    assert call(10, ctypes.c_void_p(0x100008)) == INVALID


def test_reduced_pv_kmajor_validation():
    f = rmm.lib.rmm_reduced_pv_kmajor
    base = [P, P, P, 1, 4, 2, 64, 96, 128, 48, 64, 1, P, NULL]

    def call(i, v):
        a = list(base)
        a[i] = v
        return f(*a)

    for i in (0, 1, 2, 12):
        assert call(i, NULL) == INVALID
    assert call(5, 3) == INVALID              # H % Hkv
    assert call(9, 0) == INVALID              # kt
    assert call(9, 97) == INVALID
    assert call(10, 60) == INVALID            # ldpt < Lq
    assert call(10, 68) == UNSUPPORTED        # ldpt % 8


@pytest.mark.parametrize("entry", ["rmm_decode_step", "rmm_decode_products"])
def test_decode_step_validation(entry):
    """Both grouped decode entry points validate the same way (the products
    alone take the same groups and workspace)."""
    G = rmm.DecodeGroup
    f = getattr(rmm.lib, entry)

    def arr(**kw):
        d = dict(X=0x100000, W=0x100000, idx=0x100000, Y=0x100000, K=4096, N=1024, k=2048,
                 ldx=4096, ldw=1024, ldy=1024)
        d.update(kw)
        return (G * 1)(G(**d))

    assert f(None, 1, 1, NULL, 0, NULL) == INVALID
    assert f(arr(), 0, 1, NULL, 0, NULL) == INVALID
    assert f(arr(), 1, 0, NULL, 0, NULL) == INVALID
    assert f(arr(X=None), 1, 1, NULL, 0, NULL) == INVALID
    assert f(arr(k=0), 1, 1, NULL, 0, NULL) == INVALID
    assert f(arr(k=4097), 1, 1, NULL, 0, NULL) == INVALID
    assert f(arr(ldw=1000), 1, 1, NULL, 0, NULL) == INVALID
    # wider than the one-pass token selection: accepted (its own selection
    # launch), so the missing workspace is what is reported
    assert f(arr(K=20000, ldx=20000), 1, 1, NULL, 0, NULL) == WS_SMALL
    assert f(arr(X=0x100008), 1, 1, NULL, 0, NULL) == UNSUPPORTED
    nine = (G * 9)(*[arr()[0]] * 9)
    assert f(nine, 9, 1, NULL, 0, NULL) == UNSUPPORTED
    need = rmm.lib.rmm_decode_step_workspace_size(arr(), 1, 1)
    assert need > 0                                    # one token: the list is split over slices
    assert f(arr(), 1, 1, NULL, 0, NULL) == WS_SMALL
    assert f(arr(), 1, 1, P, need - 1, NULL) == WS_SMALL


@pytest.mark.parametrize("entry", ["rmm_decode_products_shared", "rmm_decode_step_shared"])
def test_decode_products_shared_validation(entry):
    """The shared-rows products (alone, or after the step's selection)
    validate their groups as the other decode entry points do, take at most
    32 sequences, and always need workspace."""
    G = rmm.DecodeGroup
    f = getattr(rmm.lib, entry)
    size = rmm.lib.rmm_decode_products_shared_workspace_size

    def arr(**kw):
        d = dict(X=0x100000, W=0x100000, idx=0x100000, Y=0x100000, K=4096, N=1024, k=2048,
                 ldx=4096, ldw=1024, ldy=1024)
        d.update(kw)
        return (G * 1)(G(**d))

    assert f(None, 1, 1, NULL, 0, NULL) == INVALID
    assert f(arr(), 0, 1, NULL, 0, NULL) == INVALID
    assert f(arr(), 1, 0, NULL, 0, NULL) == INVALID
    assert f(arr(Y=None), 1, 1, NULL, 0, NULL) == INVALID
    assert f(arr(k=4097), 1, 1, NULL, 0, NULL) == INVALID
    assert f(arr(ldy=1000), 1, 1, NULL, 0, NULL) == INVALID
    assert f(arr(W=0x100008), 1, 1, NULL, 0, NULL) == UNSUPPORTED
    assert f(arr(ldw=1028, N=1028, ldy=1028), 1, 1, NULL, 0, NULL) == UNSUPPORTED
    assert f(arr(), 1, 33, NULL, 0, NULL) == UNSUPPORTED
    assert size(arr(), 1, 33) == 0
    nine = (G * 9)(*[arr()[0]] * 9)
    assert f(nine, 9, 1, NULL, 0, NULL) == UNSUPPORTED
    # 8 ranges of 512 indices: boundaries, union rows, counts, activations
    # and the fp32 partials of every range, each 256-byte aligned
    B, R, N = 16, 8, 1024
    a256 = lambda x: (x + 255) // 256 * 256
    want = (a256(B * (R + 1) * 4) + a256(R * 512 * 4) + a256(R * 4) + a256(R * 32 * 512 * 2)
            + a256(B * R * N * 4))
    need = size(arr(), 1, B)
    assert need == want
    assert size(arr(K=512, ldx=512, k=100), 1, B) > 0      # one range: no partials, still lists
    assert f(arr(), 1, B, NULL, 0, NULL) == WS_SMALL
    assert f(arr(), 1, B, P, need - 1, NULL) == WS_SMALL
    assert f(arr(), 1, B, ctypes.c_void_p(0x100010), need, NULL) == INVALID   # misaligned


def test_reduced_qk_rowstats_validation():
    f = rmm.lib.rmm_reduced_qk_rowstats
    # Q, Kc, idx, batch, H, Hkv, Lq, Lk, D, k, scale, causal, S, row_max, row_rinv, stream
    base = [P, P, P, 1, 4, 2, 64, 96, 128, 64, 0.125, 1, P, P, P, NULL]

    def call(i, v):
        a = list(base)
        a[i] = v
        return f(*a)

    for i in (0, 1, 2, 12, 13, 14):
        assert call(i, NULL) == INVALID
    assert call(5, 3) == INVALID              # H % Hkv
    assert call(9, 0) == INVALID              # k
    assert call(9, 129) == INVALID
    assert call(8, 96) == UNSUPPORTED         # D not 64 or 128
    assert call(7, 100) == UNSUPPORTED        # Lk % 8
    assert call(12, ctypes.c_void_p(0x100008)) == UNSUPPORTED   # S not 16-byte aligned
    assert call(13, ctypes.c_void_p(0x100002)) == UNSUPPORTED   # misaligned statistics


def test_attention_weights_kmajor_rowstats_validation():
    f = rmm.lib.rmm_attention_weights_kmajor_rowstats
    need = rmm.rmm_attention_weights_kmajor_workspace_size(1, 2, 64, 96)
    # S, batch, H, Lq, Lk, lds, causal, row_max, row_rinv, Pt, ldpt, energy, ws, bytes, stream
    base = [P, 1, 2, 64, 96, 96, 1, P, P, P, 64, P, P, need, NULL]

    def call(i, v):
        a = list(base)
        a[i] = v
        return f(*a)

    for i in (0, 7, 8, 9, 11):
        assert call(i, NULL) == INVALID
    assert call(5, 90) == INVALID             # lds < Lk
    assert call(10, 60) == INVALID            # ldpt < Lq
    assert call(5, 100) == UNSUPPORTED        # lds % 8
    assert call(8, ctypes.c_void_p(0x100002)) == UNSUPPORTED   # misaligned statistics
    assert call(12, NULL) == WS_SMALL
    assert call(13, need - 1) == WS_SMALL
    assert call(12, ctypes.c_void_p(0x100008)) == INVALID
