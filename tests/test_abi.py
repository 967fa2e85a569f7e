"""CPU checks of the C ABI: the library loads, exports every function that
include/lt.h declares, and rejects bad arguments on the host before any GPU
work (these paths make no HIP call, so they run without a GPU)."""

import ctypes

import pytest

from paper_2606_10415_amd import lt


def test_every_declared_symbol_is_exported():
    names = lt.declared_functions()
    assert {"lt_gemm_f16", "lt_gemm_f16_res", "lt_attn_fwd", "lt_attn_bwd",
            "lt_attn_bwd_workspace_size", "lt_swiglu_fwd", "lt_swiglu_bwd",
            "lt_status_string", "lt_last_error", "lt_version", "lt_rmsnorm_fwd",
            "lt_rmsnorm_bwd", "lt_rmsnorm_bwd_workspace_size", "lt_rope_table",
            "lt_rope_f16", "lt_gemm_gu_swiglu_f16", "lt_gemm_swiglu_bwd_f16", "lt_gemm_f16_bias",
            "lt_bias_grad_workspace_size", "lt_bias_grad_f16", "lt_gemm_f16_workspace_size",
            "lt_gemm_f16_ws", "lt_gemm_f16_noalloc"} <= set(names)
    for n in names:
        assert hasattr(lt._lib, n), f"{n} declared in lt.h but not exported"
    with open(lt.HEADER) as f:
        assert "#define LT_GEMM_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)" in f.read()
    assert lt.LT_GEMM_NOALLOC_SCRATCH_BYTES == 64 << 20


def test_status_strings():
    assert lt.status_string(lt.LT_OK) == "LT_OK"
    assert lt.status_string(lt.LT_ERR_INVALID_ARG) == "LT_ERR_INVALID_ARG"
    assert lt.status_string(lt.LT_ERR_UNSUPPORTED) == "LT_ERR_UNSUPPORTED"
    assert lt.status_string(lt.LT_ERR_WORKSPACE) == "LT_ERR_WORKSPACE"
    assert lt.status_string(lt.LT_ERR_HIP) == "LT_ERR_HIP"
    assert lt.status_string(99) == "LT_ERR_UNKNOWN"
    assert lt.lt_version() >= 100


FAKE = 0x1000_0000   # 16-byte aligned address that is never dereferenced (host-side rejection)


def _gemm(**kw):
    a = dict(transA=0, transB=1, M=64, N=64, K=64, alpha=1.0, A=FAKE, lda=64, B=FAKE, ldb=64,
             beta=0.0, C=FAKE, ldc=64)
    a.update(kw)
    return lt._lib.lt_gemm_f16(a["transA"], a["transB"], a["M"], a["N"], a["K"], a["alpha"], a["A"],
                               a["lda"], a["B"], a["ldb"], a["beta"], a["C"], a["ldc"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(transA=2), lt.LT_ERR_INVALID_ARG),
    (dict(M=-1), lt.LT_ERR_INVALID_ARG),
    (dict(A=None), lt.LT_ERR_INVALID_ARG),
    (dict(C=None), lt.LT_ERR_INVALID_ARG),
    (dict(lda=32), lt.LT_ERR_INVALID_ARG),
    (dict(ldc=8), lt.LT_ERR_INVALID_ARG),
    (dict(ldc=68), lt.LT_ERR_UNSUPPORTED),
    (dict(M=(1 << 30) + 8), lt.LT_ERR_UNSUPPORTED),
    (dict(lda=68), lt.LT_ERR_UNSUPPORTED),
    (dict(A=FAKE + 2), lt.LT_ERR_UNSUPPORTED),
])
def test_gemm_rejects_on_host(kw, status):
    assert _gemm(**kw) == status
    assert lt.last_error() != ""


def test_gemm_empty_is_noop():
    # M == 0 or N == 0: nothing to do, nothing launched, pointers never read
    assert _gemm(M=0, A=None, B=None, C=None) == lt.LT_OK
    assert _gemm(N=0, A=None, B=None, C=None) == lt.LT_OK


def test_gemm_res_needs_r_when_beta_nonzero():
    st = lt._lib.lt_gemm_f16_res(0, 1, 64, 64, 64, 1.0, FAKE, 64, FAKE, 64, 1.0, None, 64, FAKE, 64, None)
    assert st == lt.LT_ERR_INVALID_ARG


def _fwd(**kw):
    a = dict(Q=FAKE, K=FAKE, V=FAKE, qs=384, kvs=384, O=FAKE, os=128, LSE=FAKE, B=1, S=16, Hq=2,
             Hkv=1, D=64, scale=0.125, causal=1)
    a.update(kw)
    return lt._lib.lt_attn_fwd(a["Q"], a["K"], a["V"], a["qs"], a["kvs"], a["O"], a["os"], a["LSE"],
                               a["B"], a["S"], a["Hq"], a["Hkv"], a["D"], a["scale"], a["causal"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(Q=None), lt.LT_ERR_INVALID_ARG),
    (dict(LSE=None), lt.LT_ERR_INVALID_ARG),
    (dict(S=0), lt.LT_ERR_INVALID_ARG),
    (dict(Hq=3, Hkv=2), lt.LT_ERR_INVALID_ARG),
    (dict(causal=2), lt.LT_ERR_INVALID_ARG),
    (dict(scale=0.0), lt.LT_ERR_INVALID_ARG),
    (dict(scale=float("nan")), lt.LT_ERR_INVALID_ARG),
    (dict(qs=64), lt.LT_ERR_INVALID_ARG),
    (dict(os=64), lt.LT_ERR_INVALID_ARG),
    (dict(D=32, qs=384, os=128), lt.LT_ERR_UNSUPPORTED),
    (dict(D=96), lt.LT_ERR_UNSUPPORTED),
    (dict(qs=388), lt.LT_ERR_UNSUPPORTED),
    (dict(K=FAKE + 8), lt.LT_ERR_UNSUPPORTED),
    (dict(qs=1 << 22), lt.LT_ERR_UNSUPPORTED),          # 32-bit buffer offsets of row tiles
    (dict(kvs=1 << 22), lt.LT_ERR_UNSUPPORTED),
    (dict(os=1 << 22), lt.LT_ERR_UNSUPPORTED),
])
def test_attn_fwd_rejects_on_host(kw, status):
    assert _fwd(**kw) == status


def _align256(x):
    return (x + 255) // 256 * 256


def _ds_bytes(B, S, Hq, causal):
    n32 = (S + 31) // 32
    blocks = n32 * (n32 + 1) // 2 if causal else n32 * n32
    return _align256(B * Hq * blocks * 2048)


def test_attn_bwd_workspace():
    # D and the base-2 LSE, [B, Hq, S] fp32 each, then the fp16 dS blocks (2 KiB per
    # 32-key x 32-query pair the mask keeps), each 256-byte aligned, plus fp32 partial
    # dK, dV [2][n][B, S, Hkv, D] when a key tile's (query head, query block) pairs are
    # split n ways.  Key tiles hold 256 keys, or 128 for MHA when 256-key tiles give fewer
    # than 512 workgroups (tiles x B x Hkv); with the chosen tiles, fewer than 512
    # workgroups split n ways: the
    # smallest divisor of Hq/Hkv reaching 512 workgroups, else min(max(Hq/Hkv,
    # ceil(256 / workgroups)), 16, the last key tile's pairs).
    def rows(B, S, Hq):
        return 2 * _align256(4 * B * Hq * S)
    # MHA, S = 100: 16 workgroups, 2 query blocks in the only key tile -> n = 2
    assert lt.lt_attn_bwd_workspace_size(2, 100, 8, 8, 128, 1) == \
        rows(2, 100, 8) + _ds_bytes(2, 100, 8, 1) + _align256(2 * 2 * 2 * 100 * 8 * 128 * 4)
    # non-causal: every (key group, query group) pair
    assert lt.lt_attn_bwd_workspace_size(2, 100, 8, 8, 128, 0) == \
        rows(2, 100, 8) + _ds_bytes(2, 100, 8, 0) + _align256(2 * 2 * 2 * 100 * 8 * 128 * 4)
    assert _ds_bytes(1, 100, 1, 0) == 16 * 2048 and _ds_bytes(1, 100, 1, 1) == 10 * 2048
    # GQA 4:1, S = 100: 4 workgroups; max(4, 64) capped at 16, then at 4 heads x 2 blocks -> 8
    ws = lt.lt_attn_bwd_workspace_size(2, 100, 8, 2, 128, 1)
    assert ws == rows(2, 100, 8) + _ds_bytes(2, 100, 8, 1) + \
        _align256(2 * 8 * 2 * 100 * 2 * 128 * 4)
    assert ws % 256 == 0
    # MHA, S = 1024, 32 heads: 128-key tiles, 256 workgroups -> n = 1, no partials
    assert lt.lt_attn_bwd_workspace_size(1, 1024, 32, 32, 128, 1) == \
        rows(1, 1024, 32) + _ds_bytes(1, 1024, 32, 1)
    # MHA, S = 512: 128 workgroups of 128 keys; the last tile has 2 query blocks -> n = 2
    assert lt.lt_attn_bwd_workspace_size(1, 512, 32, 32, 128, 1) == \
        rows(1, 512, 32) + _ds_bytes(1, 512, 32, 1) + _align256(2 * 2 * 512 * 32 * 128 * 4)
    # GQA 5:1, S = 2048: 64 workgroups of 256 keys, no divisor reaches 512 -> max(4, 5)
    assert lt.lt_attn_bwd_workspace_size(1, 2048, 40, 8, 128, 1) == \
        rows(1, 2048, 40) + _ds_bytes(1, 2048, 40, 1) + _align256(2 * 5 * 2048 * 8 * 128 * 4)
    # enough kv heads x key tiles (512 or more workgroups): no split, no partials
    assert lt.lt_attn_bwd_workspace_size(1, 4096, 128, 32, 128, 1) == \
        rows(1, 4096, 128) + _ds_bytes(1, 4096, 128, 1)
    # LLaMA-2-7B heads: 32 x 8256 blocks of 2 KiB = 541 MB of dS
    assert lt.lt_attn_bwd_workspace_size(1, 4096, 32, 32, 128, 1) == \
        rows(1, 4096, 32) + 32 * 8256 * 2048
    # GQA 5:1 (Qwen2.5-32B heads), S = 4096: 128 workgroups of 256 keys, divisor 5 -> 640
    assert lt.lt_attn_bwd_workspace_size(1, 4096, 40, 8, 128, 1) == \
        rows(1, 4096, 40) + _ds_bytes(1, 4096, 40, 1) + _align256(2 * 5 * 4096 * 8 * 128 * 4)
    assert lt.lt_attn_bwd_workspace_size(1, 100, 8, 2, 128, 2) == 0
    assert lt.lt_attn_bwd_workspace_size(0, 100, 8, 2, 128, 1) == 0
    assert lt.lt_attn_bwd_workspace_size(1, 100, 8, 3, 128, 1) == 0
    args = [FAKE, FAKE, FAKE, 1536, 1536, FAKE, FAKE, 1024, FAKE, FAKE, FAKE, FAKE, 1536, 1536]
    st = lt._lib.lt_attn_bwd(*args, FAKE, ws - 1, 2, 100, 8, 2, 128, 0.09, 1, None)
    assert st == lt.LT_ERR_WORKSPACE
    st = lt._lib.lt_attn_bwd(*args, None, ws, 2, 100, 8, 2, 128, 0.09, 1, None)
    assert st == lt.LT_ERR_WORKSPACE
    st = lt._lib.lt_attn_bwd(*args, FAKE + 16, ws, 2, 100, 8, 2, 128, 0.09, 1, None)
    assert st == lt.LT_ERR_WORKSPACE
    for i in (3, 4, 7, 12, 13):                       # q, kv, o, dq, dkv row strides
        big = list(args)
        big[i] = 1 << 22
        st = lt._lib.lt_attn_bwd(*big, FAKE, ws, 2, 100, 8, 2, 128, 0.09, 1, None)
        assert st == lt.LT_ERR_UNSUPPORTED, i


def test_swiglu_rejects_on_host():
    assert lt._lib.lt_swiglu_fwd(FAKE, FAKE, 4, 12, None) == lt.LT_ERR_UNSUPPORTED
    assert lt._lib.lt_swiglu_fwd(None, FAKE, 4, 16, None) == lt.LT_ERR_INVALID_ARG
    assert lt._lib.lt_swiglu_bwd(FAKE, FAKE, FAKE, -1, 16, None) == lt.LT_ERR_INVALID_ARG
    assert lt._lib.lt_swiglu_fwd(None, None, 0, 16, None) == lt.LT_OK


def test_binding_refuses_host_tensors():
    torch = pytest.importorskip("torch")
    x = torch.zeros(8, 8, dtype=torch.float16)
    with pytest.raises(TypeError):
        lt.lt_swiglu_fwd(x, x, 8, 4)


def test_errors_raise_lt_error():
    with pytest.raises(lt.LtError) as e:
        lt.lt_gemm_f16(0, 1, -1, 8, 8, 1.0, FAKE, 8, FAKE, 8, 0.0, FAKE, 8, stream=0)
    assert e.value.status == lt.LT_ERR_INVALID_ARG


def _rms_fwd(**kw):
    a = dict(X=FAKE, ldx=4096, W=FAKE, Y=FAKE, ldy=4096, RSTD=FAKE, T=16, H=4096, eps=1e-5)
    a.update(kw)
    return lt._lib.lt_rmsnorm_fwd(a["X"], a["ldx"], a["W"], a["Y"], a["ldy"], a["RSTD"], a["T"],
                                  a["H"], a["eps"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(X=None), lt.LT_ERR_INVALID_ARG),
    (dict(H=0), lt.LT_ERR_INVALID_ARG),
    (dict(T=-1), lt.LT_ERR_INVALID_ARG),
    (dict(ldx=132, H=128), lt.LT_ERR_UNSUPPORTED),     # stride not a multiple of 8
    (dict(ldy=64, H=128), lt.LT_ERR_INVALID_ARG),      # stride below the row
    (dict(H=12, ldx=16, ldy=16), lt.LT_ERR_UNSUPPORTED),
    (dict(H=16384, ldx=16384, ldy=16384), lt.LT_ERR_UNSUPPORTED),
    (dict(eps=-1.0), lt.LT_ERR_INVALID_ARG),
    (dict(eps=float("nan")), lt.LT_ERR_INVALID_ARG),
    (dict(Y=FAKE + 8), lt.LT_ERR_UNSUPPORTED),
])
def test_rmsnorm_fwd_rejects_on_host(kw, status):
    assert _rms_fwd(**kw) == status
    assert lt.last_error()


def test_rmsnorm_empty_is_noop_and_workspace():
    assert _rms_fwd(T=0) == lt.LT_OK
    ws = lt.lt_rmsnorm_bwd_workspace_size(4096, 4096)
    # min(ceil(T / 4), 512) = 512 workgroups x one FP32 row of H partial sums
    assert ws == 512 * 4096 * 4
    assert lt.lt_rmsnorm_bwd_workspace_size(77, 5120) == 20 * 5120 * 4     # ceil(77 / 4) rows
    assert lt.lt_rmsnorm_bwd_workspace_size(3, 8) % 256 == 0
    assert lt.lt_rmsnorm_bwd_workspace_size(0, 8) == 0
    st = lt._lib.lt_rmsnorm_bwd(FAKE, 4096, FAKE, 4096, FAKE, FAKE, None, 0, FAKE, 4096, FAKE,
                                FAKE, ws - 1, 4096, 4096, None)
    assert st == lt.LT_ERR_WORKSPACE
    st = lt._lib.lt_rmsnorm_bwd(FAKE, 4096, FAKE, 4096, FAKE, FAKE, FAKE + 8, 4096, FAKE, 4096,
                                FAKE, FAKE, ws, 4096, 4096, None)
    assert st == lt.LT_ERR_UNSUPPORTED                 # misaligned residual


@pytest.mark.parametrize("args,status", [
    ((None, 16, 128, 1e4), lt.LT_ERR_INVALID_ARG),
    ((FAKE, 0, 128, 1e4), lt.LT_ERR_INVALID_ARG),
    ((FAKE, 16, 24, 1e4), lt.LT_ERR_UNSUPPORTED),      # D not a multiple of 16
    ((FAKE, 16, 128, 0.0), lt.LT_ERR_INVALID_ARG),
    ((FAKE, 16, 128, float("inf")), lt.LT_ERR_INVALID_ARG),
])
def test_rope_table_rejects_on_host(args, status):
    assert lt._lib.lt_rope_table(*args, None) == status


@pytest.mark.parametrize("kw,status", [
    (dict(inverse=2), lt.LT_ERR_INVALID_ARG),
    (dict(stride=1000), lt.LT_ERR_INVALID_ARG),        # below heads * D
    (dict(stride=6148), lt.LT_ERR_UNSUPPORTED),        # not a multiple of 8
    (dict(D=72, stride=72 * 40), lt.LT_ERR_UNSUPPORTED),
    (dict(B=0), lt.LT_ERR_INVALID_ARG),
    (dict(CS=None), lt.LT_ERR_INVALID_ARG),
])
def test_rope_rejects_on_host(kw, status):
    a = dict(X=FAKE, stride=6144, B=1, S=16, heads=40, D=128, CS=FAKE, inverse=0)
    a.update(kw)
    st = lt._lib.lt_rope_f16(a["X"], a["stride"], a["B"], a["S"], a["heads"], a["D"], a["CS"],
                             a["inverse"], None)
    assert st == status


@pytest.mark.parametrize("kw,status", [
    (dict(T=-8), lt.LT_ERR_INVALID_ARG),
    (dict(X=None), lt.LT_ERR_INVALID_ARG),
    (dict(A=None), lt.LT_ERR_INVALID_ARG),
    (dict(ldgu=1000), lt.LT_ERR_INVALID_ARG),         # below 2F
    (dict(lda=600), lt.LT_ERR_INVALID_ARG),           # below F
    (dict(ldx=100), lt.LT_ERR_INVALID_ARG),           # below H
    (dict(T=12), lt.LT_ERR_UNSUPPORTED),
    (dict(F=684, ldgu=1368, lda=684), lt.LT_ERR_UNSUPPORTED),
    (dict(ldw=132), lt.LT_ERR_UNSUPPORTED),
    (dict(GU=FAKE + 2), lt.LT_ERR_UNSUPPORTED),
])
def test_gemm_gu_swiglu_rejects_on_host(kw, status):
    a = dict(X=FAKE, ldx=128, Wgu=FAKE, ldw=128, GU=FAKE, ldgu=1376, A=FAKE, lda=688, T=64,
             H=128, F=688)
    a.update(kw)
    st = lt._lib.lt_gemm_gu_swiglu_f16(a["X"], a["ldx"], a["Wgu"], a["ldw"], a["GU"], a["ldgu"],
                                       a["A"], a["lda"], a["T"], a["H"], a["F"], None)
    assert st == status
    assert lt.last_error() != ""


@pytest.mark.parametrize("kw,status", [
    (dict(F=-8), lt.LT_ERR_INVALID_ARG),
    (dict(GU=None), lt.LT_ERR_INVALID_ARG),
    (dict(ldwd=600), lt.LT_ERR_INVALID_ARG),          # below F
    (dict(lddgu=1000), lt.LT_ERR_INVALID_ARG),        # below 2F
    (dict(H=60, lddy=60), lt.LT_ERR_UNSUPPORTED),
    (dict(dGU=FAKE + 4), lt.LT_ERR_UNSUPPORTED),
])
def test_gemm_swiglu_bwd_rejects_on_host(kw, status):
    a = dict(dY=FAKE, lddy=128, Wd=FAKE, ldwd=688, GU=FAKE, ldgu=1376, dGU=FAKE, lddgu=1376,
             T=64, H=128, F=688)
    a.update(kw)
    st = lt._lib.lt_gemm_swiglu_bwd_f16(a["dY"], a["lddy"], a["Wd"], a["ldwd"], a["GU"],
                                        a["ldgu"], a["dGU"], a["lddgu"], a["T"], a["H"], a["F"],
                                        None)
    assert st == status


def test_fused_swiglu_empty_is_noop():
    assert lt._lib.lt_gemm_gu_swiglu_f16(None, 8, None, 8, None, 0, None, 0, 0, 8, 8, None) == lt.LT_OK
    assert lt._lib.lt_gemm_swiglu_bwd_f16(None, 8, None, 8, None, 0, None, 0, 8, 8, 0, None) == lt.LT_OK


def test_gemm_bias_rejects_on_host():
    g = lambda **kw: lt._lib.lt_gemm_f16_bias(
        0, 1, kw.get("M", 64), 64, 64, 1.0, FAKE, 64, FAKE, 64, 0.0, None, 64, kw.get("bias", FAKE),
        FAKE, 64, None)
    assert g(bias=None) == lt.LT_ERR_INVALID_ARG
    assert g(bias=FAKE + 2) == lt.LT_ERR_UNSUPPORTED
    assert g(M=(1 << 30) + 8) == lt.LT_ERR_UNSUPPORTED    # beyond the tile grid
    assert g(M=0, bias=None) == lt.LT_OK          # empty: no-op


@pytest.mark.parametrize("kw,status", [
    (dict(T=0), lt.LT_ERR_INVALID_ARG),
    (dict(T=-1), lt.LT_ERR_INVALID_ARG),
    (dict(dY=None), lt.LT_ERR_INVALID_ARG),
    (dict(db=None), lt.LT_ERR_INVALID_ARG),
    (dict(lddy=32), lt.LT_ERR_INVALID_ARG),
    (dict(N=60, lddy=64), lt.LT_ERR_UNSUPPORTED),
    (dict(lddy=68), lt.LT_ERR_UNSUPPORTED),
    (dict(dY=FAKE + 2), lt.LT_ERR_UNSUPPORTED),
    (dict(ws=None), lt.LT_ERR_WORKSPACE),
    (dict(wsb=16), lt.LT_ERR_WORKSPACE),
    (dict(ws=FAKE + 8), lt.LT_ERR_UNSUPPORTED),
])
def test_bias_grad_rejects_on_host(kw, status):
    a = dict(dY=FAKE, lddy=64, T=100, N=64, db=FAKE, ws=FAKE, wsb=1 << 20)
    a.update(kw)
    st = lt._lib.lt_bias_grad_f16(a["dY"], a["lddy"], a["T"], a["N"], a["db"], a["ws"], a["wsb"], None)
    assert st == status


def test_bias_grad_workspace_and_empty():
    assert lt.lt_bias_grad_workspace_size(0, 64) == 0
    assert lt.lt_bias_grad_workspace_size(4096, 7168) == 64 * 7168 * 4
    assert lt.lt_bias_grad_workspace_size(1, 8) % 256 == 0
    assert lt._lib.lt_bias_grad_f16(None, 0, 5, 0, None, None, 0, None) == lt.LT_OK


# Split-K workspace of the last, at most half full, wave of 256x256 tiles (256 CUs):
# S = min(256 // tail_tiles, 8, ceil(K/64) // 8) splits (none below 2), FP32 partials
# over the tail region: S * Mt * Nt * 4 bytes.  A launch of fewer than 192 tiles is
# split whole, S = min(256 // tiles, 8, ceil(K/64) // 8) over all of M x N, when
# S = 8 or K >= 2048 * S.
@pytest.mark.parametrize("M,N,K,want", [
    (4096, 5120, 5120, 4 * 4096 * 1024 * 4),    # 16x20 tiles: 64 in the tail, columns 4096..5119
    (5120, 4096, 4096, 4 * 1024 * 4096 * 4),    # 20x16 tiles: rows 4096..5119
    (4096, 22016, 4096, 2 * 4096 * 1536 * 4),   # 16x86 tiles: 96 in the tail -> S = 2
    (22016, 4096, 4096, 2 * 1536 * 4096 * 4),   # 86x16 tiles: rows 20480..22015
    (4096, 5120, 1024, 2 * 4096 * 1024 * 4),    # 16 K-slices -> S = 2
    (4096, 5120, 512, 0),                       # 8 K-slices: too few to split
    (4096, 4096, 4096, 0),                      # whole waves only
    (4096, 7168, 5120, 0),                      # 448 tiles: last wave 3/4 full
    (1024, 1024, 8192, 8 * 1024 * 1024 * 4),    # 16 tiles, split whole: S = 8
    (2048, 4096, 4096, 2 * 2048 * 4096 * 4),    # 128 tiles, split whole: S = 2
    (2048, 4096, 1000, 0),                      # S = 2 but K < 4096: 128x128 tiles
    (2048, 2048, 2048, 0),                      # 64 tiles, S = 4, K < 8192
    (1024, 1024, 4096, 8 * 1024 * 1024 * 4),    # S = 8 at any K
    (2048, 3000, 4104, 2 * 2048 * 3000 * 4),    # 96 tiles, S = 2, ragged K >= 4096
    (256, 256, 256, 0),                         # 4 K-slices: too few to split
    (0, 5120, 5120, 0), (4096, 5120, 0, 0),
])
def test_gemm_workspace_size(M, N, K, want):
    for ta, tb in ((0, 1), (0, 0), (1, 0), (1, 1)):
        assert lt.lt_gemm_f16_workspace_size(ta, tb, M, N, K) == want


def _gemm_ws(ws, ws_bytes, M=4096, N=5120, K=5120):
    return lt._lib.lt_gemm_f16_ws(0, 1, M, N, K, 1.0, FAKE, K, FAKE, K, 0.0, None, N, None, FAKE, N,
                                  ws, ws_bytes, None)


def test_gemm_ws_rejects_on_host():
    need = lt.lt_gemm_f16_workspace_size(0, 1, 4096, 5120, 5120)
    assert _gemm_ws(FAKE, need - 16) == lt.LT_ERR_WORKSPACE
    assert _gemm_ws(FAKE + 8, need) == lt.LT_ERR_UNSUPPORTED
    assert lt._lib.lt_gemm_f16_ws(2, 1, 64, 64, 64, 1.0, FAKE, 64, FAKE, 64, 0.0, None, 64, None, FAKE,
                                  64, FAKE, 1 << 20, None) == lt.LT_ERR_INVALID_ARG
    assert lt._lib.lt_gemm_f16_ws(0, 1, 64, 64, 64, 1.0, FAKE, 64, FAKE, 64, 0.0, None, 64, FAKE + 2,
                                  FAKE, 64, None, 0, None) == lt.LT_ERR_UNSUPPORTED
