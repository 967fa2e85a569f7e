"""GPU parity of lt_gemm_f16 / lt_gemm_f16_res against the float64 oracle.

Bars (written here, derived in the design doc):
  * integer-valued inputs (|partial sums| < 2^24, exact in FP32): the FP16
    output equals RNE(oracle) bit for bit -- pins layouts, transposes, tails,
    alpha/beta and the residual operand with zero tolerance;
  * normal inputs: relative Frobenius error <= 5e-3;
  * full-size decoder-layer shapes: 1024 sampled entries per GEMM, each an
    oracle dot product of length K, same 5e-3 bound.
"""

import itertools

import numpy as np
import pytest

import oracle
from paper_2606_10415_amd.synth import normal_f16, uniform_int_f16, WORKLOADS
from conftest import rel_f

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    from paper_2606_10415_amd import lt
    return torch, lt


def _stored(x, trans):
    return np.ascontiguousarray(x.T) if trans else np.ascontiguousarray(x)


def _run(env, transA, transB, M, N, K, alpha, a, b, beta=0.0, c=None, r=None):
    torch, lt = env
    A = torch.from_numpy(_stored(a, transA)).cuda()
    B = torch.from_numpy(_stored(b, transB)).cuda()
    lda, ldb = A.shape[1], B.shape[1]
    if c is None:
        C = torch.full((M, N), float("nan"), dtype=torch.float16, device="cuda")
    else:
        C = torch.from_numpy(np.ascontiguousarray(c)).cuda()
    if r is None:
        lt.lt_gemm_f16(transA, transB, M, N, K, alpha, A, lda, B, ldb, beta, C, N)
    else:
        R = torch.from_numpy(np.ascontiguousarray(r)).cuda()
        lt.lt_gemm_f16_res(transA, transB, M, N, K, alpha, A, lda, B, ldb, beta, R, N, C, N)
    torch.cuda.synchronize()
    return C.cpu().numpy()


LAYOUTS = list(itertools.product([0, 1], [0, 1]))


@pytest.mark.parametrize("transA,transB", LAYOUTS)
@pytest.mark.parametrize("M,N,K", [(8, 8, 8), (136, 200, 72), (264, 520, 1000), (4096, 4096, 512),
                                   # a last wave of at most half the CUs runs as half-size tiles:
                                   # column split (8 x 34 tiles), row split (34 x 8), ragged edges
                                   (2048, 8704, 256), (8704, 2048, 256), (2040, 8696, 264),
                                   (8696, 2040, 264)])
def test_gemm_exact_integers_bitwise(env, transA, transB, M, N, K):
    print(f"gemm exact ints trans=({transA},{transB}) M={M} N={N} K={K}", flush=True)
    a = uniform_int_f16(1, (M, K), -2, 2)
    b = uniform_int_f16(2, (K, N), -2, 2)
    c = uniform_int_f16(3, (M, N), -8, 8)
    got = _run(env, transA, transB, M, N, K, 3.0, a, b, -2.0, c)
    ref = oracle.gemm(0, 0, 3.0, a, b, -2.0, c).astype(np.float16)
    assert np.array_equal(got.view(np.uint16), ref.view(np.uint16))


@pytest.mark.parametrize("transA,transB", LAYOUTS)
@pytest.mark.parametrize("M,N,K", [
    # >= 192 whole-wave 256x256 tiles: the 4-wave loop, whose 64-wide slices
    # run in pairs (an odd count adds a zero-filled slice) and whose unmasked
    # loads serve only slices inside K
    (4096, 3072, 320),    # 5 slices (odd), all whole
    (4000, 3112, 4104),   # 65 slices, the last 8 wide; M and N tails
    (3848, 3328, 200),    # 4 slices, the last 8 wide; M and N tails
    (4096, 3072, 8),      # a single 8-wide slice
])
def test_gemm_four_wave_slices_exact_integers_bitwise(env, transA, transB, M, N, K):
    print(f"gemm 4-wave slices trans=({transA},{transB}) M={M} N={N} K={K}", flush=True)
    a = uniform_int_f16(31, (M, K), -2, 2)
    b = uniform_int_f16(32, (K, N), -2, 2)
    c = uniform_int_f16(33, (M, N), -8, 8)
    got = _run(env, transA, transB, M, N, K, 3.0, a, b, -2.0, c)
    ref = oracle.gemm(0, 0, 3.0, a, b, -2.0, c).astype(np.float16)
    assert np.array_equal(got.view(np.uint16), ref.view(np.uint16))


@pytest.mark.parametrize("transA,transB", LAYOUTS)
def test_gemm_residual_operand_bitwise(env, transA, transB):
    M, N, K = 200, 136, 264
    a = uniform_int_f16(4, (M, K), -2, 2)
    b = uniform_int_f16(5, (K, N), -2, 2)
    r = uniform_int_f16(6, (M, N), -100, 100)
    got = _run(env, transA, transB, M, N, K, 1.0, a, b, 1.0, None, r)
    ref = oracle.gemm(0, 0, 1.0, a, b, 1.0, r).astype(np.float16)
    assert np.array_equal(got.view(np.uint16), ref.view(np.uint16))


def _padded(x, trans, fill):
    """x stored (transposed if trans) with its leading dimension rounded up to
    a multiple of 8; the padding holds `fill`."""
    st = _stored(x, trans)
    ld = -(-st.shape[1] // 8) * 8
    out = np.full((st.shape[0], ld), fill, np.float16)
    out[:, :st.shape[1]] = st
    return out


@pytest.mark.parametrize("transA,transB", LAYOUTS)
@pytest.mark.parametrize("M,N,K", [(1, 1, 1), (61, 45, 13), (130, 44, 70), (257, 263, 77),
                                   # 256x256 tiles with the ragged-K fix-up in the slice loop
                                   (3000, 4100, 515)])
def test_gemm_ragged_sizes_bitwise(env, transA, transB, M, N, K):
    """M, N, K not multiples of 8, leading dimensions padded to 8: the padding
    of A, B and R holds NaN (it must never reach a stored result), the padding
    of C a sentinel (it must not be written)."""
    torch, lt = env
    print(f"gemm ragged trans=({transA},{transB}) M={M} N={N} K={K}", flush=True)
    a = uniform_int_f16(21, (M, K), -2, 2)
    b = uniform_int_f16(22, (K, N), -2, 2)
    r = uniform_int_f16(23, (M, N), -8, 8)
    bias = uniform_int_f16(24, (N,), -4, 4)
    A = torch.from_numpy(_padded(a, transA, np.nan)).cuda()
    B = torch.from_numpy(_padded(b, transB, np.nan)).cuda()
    R = torch.from_numpy(_padded(r, 0, np.nan)).cuda()
    sentinel = np.float16(12345.0)
    C = torch.from_numpy(_padded(np.full((M, N), np.nan, np.float16), 0, sentinel)).cuda()
    Bias = torch.from_numpy(bias).cuda()
    lt.lt_gemm_f16_bias(transA, transB, M, N, K, 3.0, A, A.shape[1], B, B.shape[1], -2.0, R,
                        R.shape[1], Bias, C, C.shape[1])
    torch.cuda.synchronize()
    got = C.cpu().numpy()
    ref = (oracle.gemm(0, 0, 3.0, a, b, -2.0, r) + bias.astype(np.float64)).astype(np.float16)
    assert np.array_equal(got[:, :N].view(np.uint16), ref.view(np.uint16))
    assert (got[:, N:] == sentinel).all()


def test_gemm_beta_zero_ignores_nan_and_k_zero(env):
    torch, lt = env
    a = normal_f16(7, (64, 32))
    b = normal_f16(8, (32, 48))
    c = np.full((64, 48), np.nan, np.float16)
    got = _run(env, 0, 0, 64, 48, 32, 1.0, a, b, 0.0, c)
    assert np.isfinite(got).all()
    # K == 0: C = beta * C
    c2 = normal_f16(9, (64, 48))
    C = torch.from_numpy(c2).cuda()
    lt.lt_gemm_f16(0, 0, 64, 48, 0, 1.0, None, 0, None, 0, 0.5, C, 48)
    torch.cuda.synchronize()
    ref = (0.5 * c2.astype(np.float64)).astype(np.float16)
    assert np.array_equal(C.cpu().numpy().view(np.uint16), ref.view(np.uint16))


@pytest.mark.parametrize("transA,transB", LAYOUTS)
@pytest.mark.parametrize("M,N,K", [(256, 768, 256), (256, 256, 1376), (1376, 256, 256), (520, 1032, 688)])
def test_gemm_normal_parity(env, transA, transB, M, N, K):
    a = normal_f16(10, (M, K))
    b = normal_f16(11, (K, N), 0.02)
    c = normal_f16(12, (M, N))
    got = _run(env, transA, transB, M, N, K, 1.0, a, b, 1.0, c)
    ref = oracle.gemm(0, 0, 1.0, a, b, 1.0, c)
    assert rel_f(got, ref) <= 5e-3


def _layer_gemms(w):
    T = w.T
    return [("qkv_fwd", 0, 1, T, w.qkv_cols, w.H), ("o_fwd", 0, 1, T, w.H, w.Hq * w.D),
            ("gu_fwd", 0, 1, T, 2 * w.F, w.H), ("down_fwd", 0, 1, T, w.H, w.F),
            ("down_dgrad", 0, 0, T, w.F, w.H), ("gu_dgrad", 0, 0, T, w.H, 2 * w.F),
            ("qkv_dgrad", 0, 0, T, w.H, w.qkv_cols),
            ("down_wgrad", 1, 0, w.H, w.F, T), ("gu_wgrad", 1, 0, 2 * w.F, w.H, T),
            ("qkv_wgrad", 1, 0, w.qkv_cols, w.H, T)]


@pytest.mark.parametrize("name,transA,transB,M,N,K", _layer_gemms(WORKLOADS["llama2-7b"]))
def test_gemm_full_size_sampled(env, name, transA, transB, M, N, K):
    """LLaMA-2-7B layer GEMM shapes, the launch configuration the benchmark times."""
    print(f"gemm full-size {name} M={M} N={N} K={K}", flush=True)
    torch, lt = env
    seed = 5000 + 10 * [n for n, *_ in _layer_gemms(WORKLOADS["llama2-7b"])].index(name)
    # operands as stored: A [M,K] or [K,M]; B [K,N] or [N,K]
    a_np = normal_f16(seed, (K, M) if transA else (M, K))
    b_np = normal_f16(seed + 1, (N, K) if transB else (K, N), 0.02)
    A = torch.from_numpy(a_np).cuda()
    B = torch.from_numpy(b_np).cuda()
    C = torch.empty(M, N, dtype=torch.float16, device="cuda")
    lt.lt_gemm_f16(transA, transB, M, N, K, 1.0, A, A.shape[1], B, B.shape[1], 0.0, C, N)
    torch.cuda.synchronize()
    rng = np.random.default_rng(0)
    rows = rng.integers(0, M, 1024)
    cols = rng.integers(0, N, 1024)
    ref = oracle.gemm_entries(transA, transB, 1.0, a_np, b_np, 0.0, None, rows, cols)
    got = C.cpu().numpy()[rows, cols]
    assert rel_f(got, ref) <= 5e-3


# ---- lt_gemm_f16_ws: the last, at most half full, wave of 256x256 tiles with its
# K split over several workgroups (FP32 partials in the caller's workspace) ----

def _run_ws(env, transA, transB, M, N, K, alpha, a, b, beta, r, bias=None, inplace=False):
    torch, lt = env
    A = torch.from_numpy(_stored(a, transA)).cuda()
    B = torch.from_numpy(_stored(b, transB)).cuda()
    R = torch.from_numpy(np.ascontiguousarray(r)).cuda()
    C = R if inplace else torch.full((M, N), float("nan"), dtype=torch.float16, device="cuda")
    Bias = None if bias is None else torch.from_numpy(bias).cuda()
    need = lt.lt_gemm_f16_workspace_size(transA, transB, M, N, K)
    assert need > 0, "shape must take the split-K tail"
    ws = torch.full((need // 4,), float("nan"), dtype=torch.float32, device="cuda")   # contents unused
    lt.lt_gemm_f16_ws(transA, transB, M, N, K, alpha, A, A.shape[1], B, B.shape[1], beta, R, N,
                      Bias, C, N, ws, need)
    torch.cuda.synchronize()
    return C.cpu().numpy()


def _tail_rows(M, n=40, seed=3):
    rng = np.random.default_rng(seed)
    return np.unique(np.concatenate([rng.choice(M, n, replace=False),
                                     [0, 4095, 4096, M - 1] if M > 4096 else [0, M - 1]]))


@pytest.mark.parametrize("transA,transB", LAYOUTS)
@pytest.mark.parametrize("M,N,K,bias,inplace", [
    (4096, 5120, 2048, False, False),   # column tail (columns 4096..), S = 4
    (5120, 4096, 1024, True, False),    # row tail (rows 4096..), S = 2, bias
    (4088, 5112, 1000, False, True),    # ragged M/N/K, ragged last split, C = R in place
    (1024, 1536, 4096, True, False),    # 24 tiles, split whole (S = 8), bias
    (1000, 1544, 4136, False, True),    # 28 tiles, split whole (S = 8), ragged, in place
    (2048, 3000, 4104, False, False),   # 96 tiles, split whole (S = 2), ragged N and K
])
def test_gemm_ws_split_tail_exact_integers(env, transA, transB, M, N, K, bias, inplace):
    """Integer-valued inputs keep every FP32 partial and sum exact, so the split
    result equals RNE(oracle) bit for bit on sampled rows of head and tail."""
    print(f"gemm ws split tail trans=({transA},{transB}) M={M} N={N} K={K}", flush=True)
    a = uniform_int_f16(21, (M, K), -2, 2)
    b = uniform_int_f16(22, (K, N), -2, 2)
    r = uniform_int_f16(23, (M, N), -8, 8)
    bv = uniform_int_f16(24, (N,), -4, 4) if bias else None
    got = _run_ws(env, transA, transB, M, N, K, 3.0, a, b, -2.0, r, bv, inplace)
    rows = _tail_rows(M)
    ref = oracle.gemm(0, 0, 3.0, a[rows], b, -2.0, r[rows])
    if bias:
        ref = ref + bv.astype(np.float64)
    assert np.array_equal(got[rows].view(np.uint16), ref.astype(np.float16).view(np.uint16))


@pytest.mark.parametrize("transA,transB", LAYOUTS)
def test_gemm_ws_split_tail_normal_parity(env, transA, transB):
    M, N, K = 4096, 5120, 5120
    print(f"gemm ws split tail normal trans=({transA},{transB})", flush=True)
    a = normal_f16(31, (M, K))
    b = normal_f16(32, (K, N), 0.02)
    r = normal_f16(33, (M, N))
    got = _run_ws(env, transA, transB, M, N, K, 1.0, a, b, 1.0, r)
    rows = _tail_rows(M, 24)
    ref = oracle.gemm(0, 0, 1.0, a[rows], b, 1.0, r[rows])
    assert rel_f(got[rows], ref) <= 5e-3
    assert rel_f(got[rows][:, 4096:], ref[:, 4096:]) <= 5e-3      # the split columns alone
