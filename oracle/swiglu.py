"""Oracle SwiGLU gate of the FFN projection (test infrastructure only).

The paper names the FFN projection as one of the GEMM consumers (Sec. 4.1)
but not its activation; the evaluated models (LLaMA-2, Baichuan2, Qwen2.5;
Sec. 6.1) use a SwiGLU feed-forward, read here as

    A = silu(G) * U,          silu(x) = x * sigmoid(x),

with the fused gate/up projection output GU laid out [T, 2F]: columns
0..F-1 are the gate G, columns F..2F-1 are the up projection U.

Backward (product and chain rule, d silu/dx = s (1 + x (1 - s)), s = sigmoid(x)):

    dU = dA * silu(G)
    dG = dA * U * s * (1 + G * (1 - s))

float64 throughout.
"""

import numpy as np


def sigmoid(x):
    x = np.asarray(x, dtype=np.float64)
    # both branches of the textbook formula, chosen so exp never overflows
    out = np.empty_like(x)
    pos = x >= 0
    out[pos] = 1.0 / (1.0 + np.exp(-x[pos]))
    ex = np.exp(x[~pos])
    out[~pos] = ex / (1.0 + ex)
    return out


def silu(x):
    x = np.asarray(x, dtype=np.float64)
    return x * sigmoid(x)


def swiglu_fwd(gu):
    """gu [T, 2F]  ->  A [T, F] (float64)."""
    gu = np.asarray(gu, dtype=np.float64)
    F = gu.shape[1] // 2
    g, u = gu[:, :F], gu[:, F:]
    return silu(g) * u


def swiglu_bwd(da, gu):
    """da [T, F], gu [T, 2F]  ->  dGU [T, 2F] (float64): [dG | dU]."""
    da = np.asarray(da, dtype=np.float64)
    gu = np.asarray(gu, dtype=np.float64)
    F = gu.shape[1] // 2
    g, u = gu[:, :F], gu[:, F:]
    s = sigmoid(g)
    du = da * g * s
    dg = da * u * s * (1.0 + g * (1.0 - s))
    return np.concatenate([dg, du], axis=1)
