"""GPU parity of a pipeline stage of several layers with gradient accumulation.

Three layers of the tiny workload, two micro-batches in 1F1B order, weight
gradients accumulated through the GEMM's beta = 1 input.  Against the float64
oracle chained over the layers and summed over the micro-batches: every
layer's four weight gradients and both micro-batches' input gradients within
relative Frobenius error 1e-2 (three fp16-chained layers).  The full-save and
checkpointed (recompute) policies give bitwise identical results.
"""

import numpy as np
import pytest

import oracle
from paper_2606_10415_amd.synth import WORKLOADS, normal_f16
from conftest import rel_f

pytestmark = pytest.mark.gpu


def _weights(w, L):
    qkv = (w.Hq + 2 * w.Hkv) * w.D
    out = []
    for l in range(L):
        s = 500 + 10 * l
        out.append({"Wqkv": normal_f16(s, (qkv, w.H), 0.02), "Wo": normal_f16(s + 1, (w.H, w.Hq * w.D), 0.02),
                    "Wgu": normal_f16(s + 2, (2 * w.F, w.H), 0.02), "Wd": normal_f16(s + 3, (w.H, w.F), 0.02)})
    return out


def _oracle(w, weights, xs, dys):
    sh = oracle.LayerShape(w.B, w.S, w.H, w.Hq, w.Hkv, w.D, w.F)
    L = len(weights)
    dW = [{k: 0.0 for k in ("dWqkv", "dWo", "dWgu", "dWd")} for _ in range(L)]
    dxs = []
    for x, dy in zip(xs, dys):
        inputs, acts = [], []
        h = x.astype(np.float64)
        for p in weights:
            inputs.append(h)
            a = oracle.layer_fwd(sh, h, p["Wqkv"], p["Wo"], p["Wgu"], p["Wd"])
            acts.append(a)
            h = a["Y"]
        g = dy.astype(np.float64)
        for l in reversed(range(L)):
            p = weights[l]
            gr = oracle.layer_bwd(sh, inputs[l], p["Wqkv"], p["Wo"], p["Wgu"], p["Wd"], g, acts[l])
            for k in dW[l]:
                dW[l][k] = dW[l][k] + gr[k]
            g = gr["dX"]
        dxs.append(g)
    return dW, dxs


def test_stage_accumulation_matches_oracle_and_policies_agree():
    import torch
    from paper_2606_10415_amd.stage import Stage
    w = WORKLOADS["tiny"]
    L, A = 3, 2
    weights = _weights(w, L)
    xs = [normal_f16(600 + m, (w.T, w.H)) for m in range(A)]
    dys = [normal_f16(700 + m, (w.T, w.H)) for m in range(A)]
    dW_ref, dx_ref = _oracle(w, weights, xs, dys)
    got = {}
    for act in ("full", "ckpt"):
        print(f"stage L={L} A={A} act={act}", flush=True)
        st = Stage(w, L, act=act, weights=[{k: torch.from_numpy(v) for k, v in p.items()} for p in weights])
        X = [torch.from_numpy(x).cuda() for x in xs]
        dY = [torch.from_numpy(d).cuda() for d in dys]
        dx = []
        for m in range(A):
            g = st.micro_batch(X[m], dY[m], first=(m == 0))
            torch.cuda.synchronize()
            dx.append(g.cpu().numpy())
        dW = [{k: getattr(st.layers[l], k).cpu().numpy() for k in ("dWqkv", "dWo", "dWgu", "dWd")}
              for l in range(L)]
        got[act] = (dx, dW)
        errs = [rel_f(dx[m], dx_ref[m]) for m in range(A)]
        errs += [rel_f(dW[l][k], dW_ref[l][k]) for l in range(L) for k in dW[l]]
        print(f"  max error {max(errs):.3e}", flush=True)
        assert max(errs) <= 1e-2
    for m in range(A):
        assert np.array_equal(got["full"][0][m].view(np.uint16), got["ckpt"][0][m].view(np.uint16))
    for l in range(L):
        for k in got["full"][1][l]:
            assert np.array_equal(got["full"][1][l][k].view(np.uint16), got["ckpt"][1][l][k].view(np.uint16))
