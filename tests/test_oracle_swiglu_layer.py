"""Pins for the oracle SwiGLU and the composed decoder layer (CPU only).

SwiGLU: hand-derived values (tests/golden/swiglu_worked_example.json),
limits of silu, and central finite differences.  Layer: central finite
differences of L = sum(Y * dY) w.r.t. X and all four weights on a tiny GQA
layer, plus a planted mistake (residual dropped from dX) that they reject.
"""

import math

import numpy as np
import pytest

from oracle import silu, swiglu_fwd, swiglu_bwd, LayerShape, layer_fwd, layer_bwd
from paper_2606_10415_amd.synth import normal_f16
from conftest import load_golden, golden_value


def test_swiglu_worked_example():
    g = load_golden("swiglu_worked_example.json")
    G = np.array([golden_value(e) for e in g["G"]])
    U = np.full(3, golden_value(g["U"]))
    dA = np.full(3, golden_value(g["dA"]))
    gu = np.concatenate([G, U])[None, :].reshape(1, 6)
    a = swiglu_fwd(gu)[0]
    dgu = swiglu_bwd(dA[None, :], gu)[0]
    ex = g["expected"]
    np.testing.assert_allclose(a, [golden_value(e) for e in ex["A"]], rtol=1e-15, atol=1e-15)
    np.testing.assert_allclose(dgu[3:], [golden_value(e) for e in ex["dU"]], rtol=1e-15, atol=1e-15)
    np.testing.assert_allclose(dgu[:3], [golden_value(e) for e in ex["dG"]], rtol=1e-15, atol=1e-15)


def test_silu_limits():
    assert silu(np.array([0.0]))[0] == 0.0
    big = np.array([40.0, 80.0, 700.0])
    np.testing.assert_allclose(silu(big), big, rtol=1e-15)
    assert np.all(np.abs(silu(-big)) < 1e-15)
    assert np.isfinite(silu(np.array([-1e4, 1e4]))).all()


def test_swiglu_finite_differences():
    T, F = 3, 5
    gu = normal_f16(7, (T, 2 * F), 2.0).astype(np.float64)
    da = normal_f16(8, (T, F)).astype(np.float64)
    dgu = swiglu_bwd(da, gu)
    h = 1e-6
    fd = np.zeros_like(gu)
    for idx in np.ndindex(*gu.shape):
        p = gu.copy(); p[idx] += h
        m = gu.copy(); m[idx] -= h
        fd[idx] = ((swiglu_fwd(p) * da).sum() - (swiglu_fwd(m) * da).sum()) / (2 * h)
    np.testing.assert_allclose(dgu, fd, rtol=1e-7, atol=1e-8)


SHAPE = LayerShape(B=2, S=6, H=16, Hq=4, Hkv=2, D=4, F=24)


def _layer_params(seed=0):
    sh = SHAPE
    X = normal_f16(seed + 1, (sh.T, sh.H)).astype(np.float64)
    dY = normal_f16(seed + 2, (sh.T, sh.H)).astype(np.float64)
    W = {
        "Wqkv": normal_f16(seed + 3, (sh.qkv_cols, sh.H), 0.3).astype(np.float64),
        "Wo": normal_f16(seed + 4, (sh.H, sh.Hq * sh.D), 0.3).astype(np.float64),
        "Wgu": normal_f16(seed + 5, (2 * sh.F, sh.H), 0.3).astype(np.float64),
        "Wd": normal_f16(seed + 6, (sh.H, sh.F), 0.3).astype(np.float64),
    }
    return X, dY, W


def _layer_fd(grad_fn):
    sh = SHAPE
    X, dY, W = _layer_params()
    grads = grad_fn(sh, X, W["Wqkv"], W["Wo"], W["Wgu"], W["Wd"], dY)

    def loss():
        return float((layer_fwd(sh, X, W["Wqkv"], W["Wo"], W["Wgu"], W["Wd"])["Y"] * dY).sum())

    h = 1e-6
    worst = 0.0
    rng = np.random.default_rng(5)
    for name, arr in (("dX", X), ("dWqkv", W["Wqkv"]), ("dWo", W["Wo"]), ("dWgu", W["Wgu"]), ("dWd", W["Wd"])):
        flat = arr.reshape(-1)
        idxs = rng.choice(flat.size, size=min(flat.size, 60), replace=False)
        fd, an = [], []
        for t in idxs:
            old = flat[t]
            flat[t] = old + h; lp = loss()
            flat[t] = old - h; lm = loss()
            flat[t] = old
            fd.append((lp - lm) / (2 * h))
            an.append(grads[name].reshape(-1)[t])
        fd, an = np.array(fd), np.array(an)
        worst = max(worst, float(np.linalg.norm(fd - an) / np.linalg.norm(fd)))
    return worst


def test_layer_finite_differences():
    assert _layer_fd(layer_bwd) <= 1e-6


def test_planted_layer_mistake_fails_fd():
    def broken(sh, X, Wqkv, Wo, Wgu, Wd, dY):
        g = layer_bwd(sh, X, Wqkv, Wo, Wgu, Wd, dY)
        g = dict(g)
        g["dX"] = g["dX"] - g["dH1"]        # forgets the residual path of dX
        return g
    assert _layer_fd(broken) > 1e-3
