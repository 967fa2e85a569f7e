"""GPU parity of the SwiGLU kernels, the GEMMs with SwiGLU epilogues and of
the chained decoder layer.

Bars: SwiGLU outputs relative Frobenius error <= 5e-3 (per op, same fp16
inputs); the fused gate/up GEMM's GU bitwise equal to the plain GEMM's (same
tiles, same reduction order) and its A, the fused down-dgrad's dGU <= 5e-3
against the oracle (sampled rows at full size); chained layer (one fp16 input set, the GPU keeps fp16
intermediates, the oracle keeps float64 throughout): Y, dX and the four
weight gradients <= 5e-3, dQKV <= 1e-2.
"""

import numpy as np
import pytest

import oracle
from paper_2606_10415_amd.synth import normal_f16, layer_inputs, WORKLOADS, Workload
from conftest import rel_f

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    from paper_2606_10415_amd import lt
    return torch, lt


@pytest.mark.parametrize("T,F", [(256, 688), (1, 8), (37, 104), (4096, 11008)])
def test_swiglu_parity(env, T, F):
    print(f"swiglu T={T} F={F}", flush=True)
    torch, lt = env
    gu = normal_f16(31, (T, 2 * F), 2.0)
    da = normal_f16(32, (T, F))
    GU = torch.from_numpy(gu).cuda()
    dA = torch.from_numpy(da).cuda()
    A = torch.empty(T, F, dtype=torch.float16, device="cuda")
    dGU = torch.empty(T, 2 * F, dtype=torch.float16, device="cuda")
    lt.lt_swiglu_fwd(GU, A, T, F)
    lt.lt_swiglu_bwd(dA, GU, dGU, T, F)
    torch.cuda.synchronize()
    assert rel_f(A.cpu().numpy(), oracle.swiglu_fwd(gu)) <= 5e-3
    assert rel_f(dGU.cpu().numpy(), oracle.swiglu_bwd(da, gu)) <= 5e-3


def test_swiglu_extreme_inputs(env):
    torch, lt = env
    g = np.array([[-1e4, -90.0, -20.0, 0.0, 20.0, 90.0, 1e4, -0.0]], np.float16)
    gu = np.concatenate([g, np.ones_like(g)], axis=1)
    GU = torch.from_numpy(gu).cuda()
    A = torch.empty(1, 8, dtype=torch.float16, device="cuda")
    dGU = torch.empty(1, 16, dtype=torch.float16, device="cuda")
    lt.lt_swiglu_fwd(GU, A, 1, 8)
    lt.lt_swiglu_bwd(torch.ones(1, 8, dtype=torch.float16, device="cuda"), GU, dGU, 1, 8)
    torch.cuda.synchronize()
    a = A.cpu().numpy().astype(np.float64)
    assert np.isfinite(a).all() and np.isfinite(dGU.cpu().numpy()).all()
    np.testing.assert_allclose(a, oracle.swiglu_fwd(gu), rtol=2e-3, atol=1e-6)


@pytest.mark.parametrize("T,H,F", [(272, 256, 344), (64, 128, 688), (8, 64, 8), (1000, 512, 1000),
                                   (4096, 4096, 11008), (2048, 5120, 13824),
                                   (2040, 512, 5000),
                                   # half-size tail tiles: column split of both epilogues,
                                   # row split of both, and ragged versions
                                   (2048, 256, 8704), (8704, 256, 2048), (2040, 256, 8696),
                                   (8696, 256, 2040)])
def test_fused_gemm_swiglu_parity(env, T, H, F):
    print(f"fused gemm swiglu T={T} H={H} F={F}", flush=True)
    torch, lt = env
    x = normal_f16(61, (T, H))
    wgu = normal_f16(62, (2 * F, H), 0.02)
    dy = normal_f16(63, (T, H))
    wd = normal_f16(64, (H, F), 0.02)
    cu = lambda a: torch.from_numpy(a).cuda()
    X, Wgu, dY, Wd = cu(x), cu(wgu), cu(dy), cu(wd)
    e = lambda *s_: torch.full(s_, float("nan"), dtype=torch.float16, device="cuda")
    GU, A, GUref, dGU = e(T, 2 * F), e(T, F), e(T, 2 * F), e(T, 2 * F)
    lt.lt_gemm_gu_swiglu_f16(X, H, Wgu, H, GU, 2 * F, A, F, T, H, F)
    lt.lt_gemm_f16(0, 1, T, 2 * F, H, 1.0, X, H, Wgu, H, 0.0, GUref, 2 * F)
    lt.lt_gemm_swiglu_bwd_f16(dY, H, Wd, F, GU, 2 * F, dGU, 2 * F, T, H, F)
    torch.cuda.synchronize()
    assert torch.equal(GU.view(torch.int16), GUref.view(torch.int16))
    rows = np.arange(T) if T <= 1024 else np.unique(
        np.concatenate([np.random.default_rng(7).choice(T, 40, replace=False), [0, T - 1]]))
    gu = GU.cpu().numpy()
    gu_ref = oracle.gemm(0, 1, 1.0, x[rows], wgu)
    err_gu = rel_f(gu[rows], gu_ref)
    err_a = rel_f(A.cpu().numpy()[rows], oracle.swiglu_fwd(gu_ref))
    da_ref = oracle.gemm(0, 0, 1.0, dy[rows], wd)
    err_dgu = rel_f(dGU.cpu().numpy()[rows], oracle.swiglu_bwd(da_ref, gu[rows]))
    print(f"  GU {err_gu:.3e}  A {err_a:.3e}  dGU {err_dgu:.3e}", flush=True)
    assert err_gu <= 5e-3 and err_a <= 5e-3 and err_dgu <= 5e-3


def _chained(env, w, fuse=False):
    torch, lt = env
    from paper_2606_10415_amd.layer import DecoderLayer
    p = layer_inputs(w)
    L = DecoderLayer(w, p, fuse_swiglu=fuse)
    L.step()
    torch.cuda.synchronize()
    return p, L


@pytest.mark.parametrize("w", [WORKLOADS["tiny"],
                               Workload("tiny-gqa", 10, B=2, S=136, H=256, Hq=4, Hkv=2, D=64, F=344)],
                         ids=["tiny", "tiny-gqa-ragged"])
@pytest.mark.parametrize("fuse", [False, True], ids=["swiglu-kernels", "swiglu-fused"])
def test_layer_chained_parity(env, w, fuse):
    print(f"layer chained {w.name} fuse_swiglu={fuse}", flush=True)
    p, L = _chained(env, w, fuse)
    sh = oracle.LayerShape(w.B, w.S, w.H, w.Hq, w.Hkv, w.D, w.F)
    acts = oracle.layer_fwd(sh, p["X"], p["Wqkv"], p["Wo"], p["Wgu"], p["Wd"])
    grads = oracle.layer_bwd(sh, p["X"], p["Wqkv"], p["Wo"], p["Wgu"], p["Wd"], p["dY"], acts)
    c = lambda t: t.cpu().numpy()
    assert rel_f(c(L.Y), acts["Y"]) <= 5e-3
    assert rel_f(c(L.dX), grads["dX"]) <= 5e-3
    for name in ("dWqkv", "dWo", "dWgu", "dWd"):
        assert rel_f(c(getattr(L, name)), grads[name]) <= 5e-3, name
    assert rel_f(c(L.dQKV), grads["dQKV"]) <= 1e-2
