"""Full-size decoder layer in the launch configuration the benchmark times.

One fwd+bwd step of ``DecoderLayer`` (fused SwiGLU, the layer's default) at the
LLaMA-2-7B (MHA), Baichuan2-13B (MHA), Qwen2.5-32B (GQA 5:1) and LLaMA-2-70B
(GQA 8:1, two sequences) shapes, S = 4096.  Every step
of the layer is checked against the float64 oracle on outputs the oracle can
compute one by one, taking that step's inputs from the GPU's own buffers:
sampled rows of each activation / input-gradient product, sampled entries of
each weight gradient (full-length dot products over the T tokens), and whole
attention heads (forward O and LSE, backward dQ, dK, dV) for sampled heads of
every sequence of the micro-batch (with grouped queries, every query head of
the sampled kv head for dQ).

Bars: relative Frobenius error <= 5e-3 for GEMM outputs, SwiGLU outputs and
attention O; <= 1e-2 for dQ, dK, dV; LSE absolute error <= 1e-4.  Attention
heads also meet their bar per row (each row's error norm against the head's
RMS row norm).
"""

import numpy as np
import pytest

import oracle
from paper_2606_10415_amd.synth import WORKLOADS, layer_inputs
from conftest import rel_f, row_err

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name,heads", [("llama2-7b", (0, 31)), ("baichuan2-13b", (3, 39)),
                                        ("qwen2.5-32b", (7, 33)), ("llama2-70b", (9, 62))])
def test_full_size_layer_step_sampled(name, heads):
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    from paper_2606_10415_amd.layer import DecoderLayer
    w = WORKLOADS[name]
    print(f"full-size layer step {name}", flush=True)
    p = layer_inputs(w)
    L = DecoderLayer(w, p)
    L.step()
    torch.cuda.synchronize()
    c = lambda t: t.cpu().numpy()
    T, H, F, D = w.T, w.H, w.F, w.D
    S = w.S
    qd, kd = w.Hq * D, w.Hkv * D
    rng = np.random.default_rng(99)
    rows = np.unique(np.concatenate([rng.choice(T, 14, replace=False), [0, 1, T - 1]]))
    X, dY = p["X"], p["dY"]
    QKV, O, LSE, H1, GU, A, Y = (c(L.QKV), c(L.O), c(L.LSE), c(L.H1), c(L.GU), c(L.A), c(L.Y))
    dGU, dH1, dO, dQKV, dX = c(L.dGU), c(L.dH1), c(L.dO), c(L.dQKV), c(L.dX)
    err = {}

    def attn(name, got, ref):                          # whole head: rel_F and per-row bound
        err[name] = rel_f(got, ref)
        err[name + "_row"] = row_err(got, ref)

    def ent(tA, tB, Am, Bm, out):                      # sampled weight-gradient entries
        r = rng.integers(0, out.shape[0], 48)
        cc = rng.integers(0, out.shape[1], 48)
        return rel_f(out[r, cc], oracle.gemm_entries(tA, tB, 1.0, Am, Bm, 0.0, None, r, cc))

    # ---- forward, each step from the GPU's inputs to it ----
    err["QKV"] = rel_f(QKV[rows], oracle.gemm(0, 1, 1.0, X[rows], p["Wqkv"]))
    scale = 1.0 / np.sqrt(D)
    g = w.Hq // w.Hkv
    for bi in range(w.B):                              # every sequence of the micro-batch
        seq = slice(bi * S, (bi + 1) * S)

        def head(base, i):
            return QKV[seq, base + i * D:base + (i + 1) * D]

        for h in heads:
            kv = h // g
            q, k, v = head(0, h), head(qd, kv), head(qd + kd, kv)
            o, lse, _ = oracle.attn_head_fwd(q, k, v, scale, causal=True)
            attn(f"O[b{bi}h{h}]", O[seq, h * D:(h + 1) * D], o)
            lse_err = float(np.max(np.abs(LSE[bi, h] - lse)))
            assert lse_err <= 1e-4, (bi, h, lse_err)
            gr = oracle.attn_head_bwd(q, k, v, dO[seq, h * D:(h + 1) * D], scale, causal=True)
            attn(f"dQ[b{bi}h{h}]", dQKV[seq, h * D:(h + 1) * D], gr["dq"])
            if g == 1:     # MHA: dK, dV of this kv head come from this query head alone
                attn(f"dK[b{bi}h{h}]", dQKV[seq, qd + kv * D:qd + (kv + 1) * D], gr["dk"])
                attn(f"dV[b{bi}h{h}]", dQKV[seq, qd + kd + kv * D:qd + kd + (kv + 1) * D],
                     gr["dv"])
        if g > 1:          # GQA: the kv head's gradient sums its g query heads
            kv = heads[0] // g
            k, v = head(qd, kv), head(qd + kd, kv)
            dk = np.zeros((S, D))
            dv = np.zeros((S, D))
            for h in range(kv * g, (kv + 1) * g):
                gr = oracle.attn_head_bwd(head(0, h), k, v, dO[seq, h * D:(h + 1) * D], scale,
                                          causal=True)
                dk += gr["dk"]
                dv += gr["dv"]
                if h not in heads:
                    attn(f"dQ[b{bi}h{h}]", dQKV[seq, h * D:(h + 1) * D], gr["dq"])
            attn(f"dK[b{bi}kv{kv}]", dQKV[seq, qd + kv * D:qd + (kv + 1) * D], dk)
            attn(f"dV[b{bi}kv{kv}]", dQKV[seq, qd + kd + kv * D:qd + kd + (kv + 1) * D], dv)
    err["H1"] = rel_f(H1[rows], oracle.gemm(0, 1, 1.0, O[rows], p["Wo"], 1.0, X[rows]))
    gu = oracle.gemm(0, 1, 1.0, H1[rows], p["Wgu"])
    err["GU"] = rel_f(GU[rows], gu)
    err["A"] = rel_f(A[rows], oracle.swiglu_fwd(gu))
    err["Y"] = rel_f(Y[rows], oracle.gemm(0, 1, 1.0, A[rows], p["Wd"], 1.0, H1[rows]))
    # ---- backward ----
    err["dWd"] = ent(1, 0, dY, A, c(L.dWd))
    err["dGU"] = rel_f(dGU[rows], oracle.swiglu_bwd(oracle.gemm(0, 0, 1.0, dY[rows], p["Wd"]),
                                                    GU[rows]))
    err["dWgu"] = ent(1, 0, dGU, H1, c(L.dWgu))
    err["dH1"] = rel_f(dH1[rows], oracle.gemm(0, 0, 1.0, dGU[rows], p["Wgu"], 1.0, dY[rows]))
    err["dWo"] = ent(1, 0, dH1, O, c(L.dWo))
    err["dO"] = rel_f(dO[rows], oracle.gemm(0, 0, 1.0, dH1[rows], p["Wo"]))
    err["dWqkv"] = ent(1, 0, dQKV, X, c(L.dWqkv))
    err["dX"] = rel_f(dX[rows], oracle.gemm(0, 0, 1.0, dQKV[rows], p["Wqkv"], 1.0, dH1[rows]))
    print("  " + ", ".join(f"{k} {v:.2e}" for k, v in err.items()), flush=True)
    for k, v in err.items():
        bar = 1e-2 if k.startswith(("dQ[", "dK[", "dV[")) else 5e-3
        assert v <= bar, (k, v)
