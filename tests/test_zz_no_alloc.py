"""GPU check of lt_gemm_f16_noalloc, the allocation-free form of
lt_gemm_f16_ws (split-K partials in a static device array).

Through the C ABI it must give the same bits as lt_gemm_f16_ws with a
caller workspace, on two calls in a row (the second smaller, so stale
partials of the first would show), and on integer inputs the exact
RNE-rounded product of the float64 oracle.
"""

import numpy as np
import pytest

import oracle

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    from paper_2606_10415_amd import lt
    return torch, lt


def _operands(rng, tA, tB, M, N, K, integer):
    a_shape = (K, M) if tA else (M, K)
    b_shape = (N, K) if tB else (K, N)
    if integer:
        a = rng.integers(-2, 3, a_shape).astype(np.float16)
        b = rng.integers(-2, 3, b_shape).astype(np.float16)
    else:
        a = rng.standard_normal(a_shape, dtype=np.float32).astype(np.float16)
        b = (0.02 * rng.standard_normal(b_shape, dtype=np.float32)).astype(np.float16)
    return a, b


def _both(env, tA, tB, M, N, K, a, b, beta=0.0, r=None, bias=None):
    torch, lt = env
    A, B = torch.from_numpy(a).cuda(), torch.from_numpy(b).cuda()
    R = torch.from_numpy(r).cuda() if r is not None else None
    bi = torch.from_numpy(bias).cuda() if bias is not None else None
    need = lt.lt_gemm_f16_workspace_size(tA, tB, M, N, K)
    assert 0 < need <= lt.LT_GEMM_NOALLOC_SCRATCH_BYTES, need      # the split path is exercised
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    C_ws = torch.full((M, N), float("nan"), dtype=torch.float16, device="cuda")
    C_na = torch.full((M, N), float("nan"), dtype=torch.float16, device="cuda")
    lda, ldb = a.shape[1], b.shape[1]
    lt.lt_gemm_f16_ws(tA, tB, M, N, K, 1.0, A, lda, B, ldb, beta, R, N, bi, C_ws, N, ws, need)
    lt.lt_gemm_f16_noalloc(tA, tB, M, N, K, 1.0, A, lda, B, ldb, beta, R, N, bi, C_na, N)
    torch.cuda.synchronize()
    return C_ws.cpu().numpy(), C_na.cpu().numpy()


# (transA, transB, M, N, K): whole-launch splits (under one wave of 256x256
# tiles, 8 shares) and a last-wave split (the LLaMA-2-7B gate/up forward
# shape), each followed by a smaller call.
PAIRS = [
    ((1, 0, 1024, 1024, 8192), (1, 0, 512, 512, 4096)),
    ((0, 1, 4096, 22016, 4096), (0, 0, 1024, 4096, 22016)),
]


@pytest.mark.parametrize("first,second", PAIRS)
def test_noalloc_matches_workspace_entry_point(env, first, second):
    rng = np.random.default_rng(7)
    for i, (tA, tB, M, N, K) in enumerate((first, second)):
        print(f"noalloc call {i}: transA={tA} transB={tB} M={M} N={N} K={K}", flush=True)
        a, b = _operands(rng, tA, tB, M, N, K, integer=False)
        c_ws, c_na = _both(env, tA, tB, M, N, K, a, b)
        assert np.array_equal(c_ws.view(np.uint16), c_na.view(np.uint16))
        rows = rng.choice(M, 8, replace=False)
        ref = oracle.gemm(tA, tB, 1.0, a[:, rows] if tA else a[rows], b)
        got = c_na[rows].astype(np.float64)
        assert np.linalg.norm(got - ref) <= 5e-3 * np.linalg.norm(ref)


def test_noalloc_integer_exact_with_residual_and_bias(env):
    """Integer operands (|sums| < 2^24): every output equals RNE(oracle) bit for bit,
    with beta * R and the bias added in the split's reduction; then a smaller call."""
    rng = np.random.default_rng(11)
    for tA, tB, M, N, K in ((1, 0, 1024, 1024, 8192), (0, 0, 512, 512, 4096)):
        print(f"noalloc integer: transA={tA} transB={tB} M={M} N={N} K={K}", flush=True)
        a, b = _operands(rng, tA, tB, M, N, K, integer=True)
        r = rng.integers(-4, 5, (M, N)).astype(np.float16)
        bias = rng.integers(-3, 4, (N,)).astype(np.float16)
        c_ws, c_na = _both(env, tA, tB, M, N, K, a, b, beta=1.0, r=r, bias=bias)
        ref = oracle.gemm(tA, tB, 1.0, a, b, 1.0, r.astype(np.float64)) + bias.astype(np.float64)
        assert np.array_equal(c_na.view(np.uint16), ref.astype(np.float16).view(np.uint16))
        assert np.array_equal(c_ws.view(np.uint16), c_na.view(np.uint16))
