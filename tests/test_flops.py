"""Pins of the algorithmic FLOP counts behind every TFLOP/s figure.

Both ``oracle.layer_flops`` and ``bench.layer_flops`` are checked against
  * an independent derivation: the 12 GEMM shapes of one layer step written
    out as (M, N, K) triples from the composition (forward NT, dgrad NN,
    wgrad TN of each of the four weights), each costing 2 M N K, and the
    causal (i, j) pairs counted by brute force from the mask;
  * the per-layer work table of the measurement plan (GEMM fwd+bwd, attention
    forward = 2 contractions, attention backward = the 4 contractions of
    Algorithm 1, over the causal triangle), to its printed digits.
"""

import numpy as np
import pytest

import bench
import oracle
from paper_2606_10415_amd.synth import WORKLOADS


def gemm_shapes(w):
    """(M, N, K) of the 12 products of one layer step (Sec. 4.1 consumers:
    QKV, output and FFN projections, each forward, dgrad and wgrad)."""
    T, H, F = w.T, w.H, w.F
    weights = [(w.qkv_cols, H), (H, w.Hq * w.D), (2 * F, H), (H, F)]   # [out, in]
    shapes = []
    for out, inp in weights:
        shapes += [(T, out, inp),      # Y  = X W^T
                   (T, inp, out),      # dX = dY W
                   (out, inp, T)]      # dW = dY^T X
    return shapes


def causal_pairs(S):
    i = np.arange(S)[:, None]
    j = np.arange(S)[None, :]
    return int(np.count_nonzero(j <= i))


def derived(w):
    gemm = sum(2 * M * N * K for M, N, K in gemm_shapes(w))
    pairs = causal_pairs(w.S)
    per_pair = 2 * w.D                               # one length-d contraction of one pair
    fwd = 2 * per_pair * pairs * w.Hq * w.B          # S = Q K^T, O = P V
    bwd = 4 * per_pair * pairs * w.Hq * w.B          # GP, GV, GQ, GK
    return {"gemm": gemm, "attn_fwd": fwd, "attn_bwd": bwd, "total": gemm + fwd + bwd}


# per-layer work table, printed digits (GF for tiny, TF otherwise)
TABLE = {
    "tiny": {"gemm": 1.214e9, "attn_fwd": 33.7e6, "attn_bwd": 67.4e6, "total": 1.31e9},
    "llama2-7b": {"gemm": 4.974e12, "attn_fwd": 0.1375e12, "attn_bwd": 0.2749e12,
                  "total": 5.386e12},
    "baichuan2-13b": {"gemm": 7.747e12, "attn_fwd": 0.1718e12, "attn_bwd": 0.3437e12,
                      "total": 8.263e12},
    "qwen2.5-32b": {"gemm": 11.98e12, "attn_fwd": 0.1718e12, "attn_bwd": 0.3437e12,
                    "total": 12.50e12},
    "llama2-70b": {"gemm": 42.06e12, "attn_fwd": 0.5499e12, "attn_bwd": 1.0998e12,
                   "total": 43.71e12},
}


def _oracle_flops(w):
    sh = oracle.LayerShape(w.B, w.S, w.H, w.Hq, w.Hkv, w.D, w.F)
    return oracle.layer_flops(sh)


@pytest.mark.parametrize("name", list(WORKLOADS))
def test_flops_match_independent_derivation(name):
    w = WORKLOADS[name]
    ref = derived(w)
    assert bench.layer_flops(w) == ref
    assert _oracle_flops(w) == ref


@pytest.mark.parametrize("name", list(TABLE))
def test_flops_match_work_table(name):
    w = WORKLOADS[name]
    for f in (bench.layer_flops(w), _oracle_flops(w)):
        for key, printed in TABLE[name].items():
            digits = len(f"{printed:.4g}".replace(".", "").lstrip("0").split("e")[0])
            assert f[key] == pytest.approx(printed, rel=0.6 * 10.0 ** (1 - digits)), (name, key)


def test_llama2_7b_exact_total():
    # 6 T H (2H + 2 Hkv d + 3F) + 12 d S(S+1)/2 Hq B at T = S = H = 4096,
    # Hq = Hkv = 32, d = 128, F = 11008, B = 1
    assert bench.layer_flops(WORKLOADS["llama2-7b"])["total"] == 5_385_989_652_480


def test_planted_mistake_is_caught():
    """A count that drops the causal diagonal (S(S-1)/2 pairs) must differ."""
    w = WORKLOADS["tiny"]
    wrong = 4 * 2 * w.D * (w.S * (w.S - 1) // 2) * w.Hq * w.B
    assert wrong != derived(w)["attn_bwd"]
