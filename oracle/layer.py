"""Oracle decoder layer forward + backward (test infrastructure only).

Composition of the oracle steps into one dense decoder layer as used by the
paper's workloads (decoder-only Transformer layers, Sec. 2.2 and Sec. 3.3;
GEMM consumers QKV / output / FFN projections, Sec. 4.1; LLaMA-2, Baichuan2,
Qwen2.5 shapes, Sec. 6.1).  The paper mentions no normalisation, rotary
embedding, bias or dropout, so the layer here has none; the two residual
additions are kept.

Forward, X [T, H] with T = B*S rows (batch-major):
    QKV = X Wqkv^T          Wqkv [(Hq + 2 Hkv) d, H]: Q heads, then K, then V
    O, LSE = attention(Q, K, V)   per batch, causal
    H1  = X + O Wo^T         Wo  [H, Hq d]
    GU  = H1 Wgu^T           Wgu [2F, H]: gate rows, then up rows
    A   = silu(G) * U
    Y   = H1 + A Wd^T        Wd  [H, F]

Backward of sum(Y * dY):
    dWd = dY^T A ;  dA = dY Wd ;  dGU = swiglu_bwd(dA, GU)
    dWgu = dGU^T H1 ;  dH1 = dY + dGU Wgu
    dWo = dH1^T O ;  dO = dH1 Wo
    dQ, dK, dV = attention_bwd(Q, K, V, dO) -> dQKV
    dWqkv = dQKV^T X ;  dX = dH1 + dQKV Wqkv

With ``norm`` (a LayerNorms: RMSNorm weights of the attention and FFN
inputs, eps, rotary base) the layer is the full LLaMA-2 / Qwen2.5 block of the
evaluated models (Sec. 6.1): each block's input is RMSNorm-ed and Q, K are
rotated (norm_rope.py):

    Xn  = rmsnorm(X, wn1);   QKV = Xn Wqkv^T;   Q, K <- rope(Q), rope(K)
    H1  = X + attention(Q, K, V) Wo^T
    H1n = rmsnorm(H1, wn2);  GU = H1n Wgu^T;    Y = H1 + swiglu(GU) Wd^T

and the backward adds rmsnorm_bwd after each block's input GEMM gradient
and the inverse rotation of dQ, dK before the QKV weight / data gradients.

Qwen2.5's QKV projection carries a bias (``norm.bqkv``, [(Hq + 2 Hkv) d]): it
is part of the linear layer, so it is added to QKV before the rotation, and
its gradient is the column sum of dQKV taken after the inverse rotation:

    QKV = Xn Wqkv^T + bqkv ;   dbqkv = sum over rows of dQKV

All intermediates stay float64 (no float16 rounding of intermediates).
"""

from dataclasses import dataclass

import numpy as np

from .attention import attn_fwd, attn_bwd
from .gemm import column_sum
from .norm_rope import rmsnorm_fwd, rmsnorm_bwd, rope_fwd, rope_bwd
from .swiglu import swiglu_fwd, swiglu_bwd


@dataclass(frozen=True)
class LayerShape:
    B: int      # micro-batch
    S: int      # sequence length
    H: int      # hidden size
    Hq: int     # query heads
    Hkv: int    # key/value heads
    D: int      # head dim
    F: int      # FFN size

    @property
    def T(self):
        return self.B * self.S

    @property
    def qkv_cols(self):
        return (self.Hq + 2 * self.Hkv) * self.D


@dataclass(frozen=True)
class LayerNorms:
    wn1: object          # RMSNorm weight of the attention input [H]
    wn2: object          # RMSNorm weight of the FFN input [H]
    eps: float = 1e-5
    rope_base: float = 10000.0
    bqkv: object = None  # QKV projection bias [(Hq + 2 Hkv) d] (Qwen2.5), or None


def _split_qkv(qkv, sh):
    """[T, (Hq+2Hkv)d] -> q [B,S,Hq,d], k, v [B,S,Hkv,d] (views)."""
    qd = sh.Hq * sh.D
    kd = sh.Hkv * sh.D
    q = qkv[:, :qd].reshape(sh.B, sh.S, sh.Hq, sh.D)
    k = qkv[:, qd:qd + kd].reshape(sh.B, sh.S, sh.Hkv, sh.D)
    v = qkv[:, qd + kd:].reshape(sh.B, sh.S, sh.Hkv, sh.D)
    return q, k, v


def layer_fwd(sh, X, Wqkv, Wo, Wgu, Wd, norm=None):
    """Returns a dict of float64 activations including 'Y'."""
    X = np.asarray(X, dtype=np.float64)
    Wqkv, Wo, Wgu, Wd = (np.asarray(w, dtype=np.float64) for w in (Wqkv, Wo, Wgu, Wd))
    scale = 1.0 / np.sqrt(sh.D)
    acts = {}
    Xin = X
    if norm is not None:
        Xin, acts["rstd1"] = rmsnorm_fwd(X, norm.wn1, norm.eps)
        acts["Xn"] = Xin
    qkv = Xin @ Wqkv.T
    if norm is not None and norm.bqkv is not None:
        qkv = qkv + np.asarray(norm.bqkv, dtype=np.float64)[None, :]
    q, k, v = _split_qkv(qkv, sh)
    if norm is not None:
        q, k = rope_fwd(q, norm.rope_base), rope_fwd(k, norm.rope_base)
        qkv = np.concatenate([q.reshape(sh.T, -1), k.reshape(sh.T, -1), v.reshape(sh.T, -1)], axis=1)
    o4, lse = attn_fwd(q, k, v, scale, causal=True)
    O = o4.reshape(sh.T, sh.Hq * sh.D)
    H1 = X + O @ Wo.T
    H1in = H1
    if norm is not None:
        H1in, acts["rstd2"] = rmsnorm_fwd(H1, norm.wn2, norm.eps)
        acts["H1n"] = H1in
    GU = H1in @ Wgu.T
    A = swiglu_fwd(GU)
    Y = H1 + A @ Wd.T
    acts.update({"QKV": qkv, "O": O, "LSE": lse, "H1": H1, "GU": GU, "A": A, "Y": Y})
    return acts


def layer_bwd(sh, X, Wqkv, Wo, Wgu, Wd, dY, acts=None, norm=None):
    """Gradient of sum(Y * dY) w.r.t. X and the weights (float64 dict; with
    ``norm`` also 'dWn1', 'dWn2' for the two RMSNorm weights, and 'dbqkv' when
    the norm carries a QKV bias)."""
    X = np.asarray(X, dtype=np.float64)
    Wqkv, Wo, Wgu, Wd = (np.asarray(w, dtype=np.float64) for w in (Wqkv, Wo, Wgu, Wd))
    dY = np.asarray(dY, dtype=np.float64)
    if acts is None:
        acts = layer_fwd(sh, X, Wqkv, Wo, Wgu, Wd, norm=norm)
    scale = 1.0 / np.sqrt(sh.D)
    out = {}
    dWd = dY.T @ acts["A"]
    dA = dY @ Wd
    dGU = swiglu_bwd(dA, acts["GU"])
    dWgu = dGU.T @ acts["H1n" if norm is not None else "H1"]
    dH1in = dGU @ Wgu
    if norm is not None:
        dx2, out["dWn2"] = rmsnorm_bwd(dH1in, acts["H1"], norm.wn2, norm.eps)
        dH1 = dY + dx2
    else:
        dH1 = dY + dH1in
    dWo = dH1.T @ acts["O"]
    dO = dH1 @ Wo
    q, k, v = _split_qkv(acts["QKV"], sh)
    dq, dk, dv, _ = attn_bwd(q, k, v, dO.reshape(sh.B, sh.S, sh.Hq, sh.D), scale, causal=True)
    if norm is not None:
        dq, dk = rope_bwd(dq, norm.rope_base), rope_bwd(dk, norm.rope_base)
    dQKV = np.concatenate([dq.reshape(sh.T, -1), dk.reshape(sh.T, -1), dv.reshape(sh.T, -1)], axis=1)
    if norm is not None and norm.bqkv is not None:
        out["dbqkv"] = column_sum(dQKV)
    dWqkv = dQKV.T @ (acts["Xn"] if norm is not None else X)
    dXin = dQKV @ Wqkv
    if norm is not None:
        dx1, out["dWn1"] = rmsnorm_bwd(dXin, X, norm.wn1, norm.eps)
        dX = dH1 + dx1
    else:
        dX = dH1 + dXin
    out.update({"dX": dX, "dWqkv": dWqkv, "dWo": dWo, "dWgu": dWgu, "dWd": dWd,
                "dA": dA, "dGU": dGU, "dH1": dH1, "dO": dO, "dQKV": dQKV})
    return out


def layer_flops(sh):
    """Algorithmic FLOPs (2 per multiply-add) of one layer forward + backward.

    GEMMs: every weight is used by three products (fwd, dgrad, wgrad).
    Attention counts only the causal triangle S(S+1)/2 of (i, j) pairs:
    forward 2 contractions (QK^T, PV), backward the 4 contractions of
    Algorithm 1 (GO V^T, P^T GO, GS K, GS^T Q); the score recomputation
    of a recompute-P backward is not counted.
    """
    T = sh.T
    # per weight [out, in]: forward product 2*T*out*in FLOPs
    gemm_fwd = 2 * T * (sh.qkv_cols * sh.H          # Wqkv
                        + sh.H * sh.Hq * sh.D       # Wo
                        + 2 * sh.F * sh.H           # Wgu
                        + sh.H * sh.F)              # Wd
    pairs = sh.S * (sh.S + 1) // 2
    attn_fwd_fl = 2 * 2 * sh.D * pairs * sh.Hq * sh.B
    attn_bwd_fl = 4 * 2 * sh.D * pairs * sh.Hq * sh.B
    return {"gemm": 3 * gemm_fwd, "attn_fwd": attn_fwd_fl, "attn_bwd": attn_bwd_fl,
            "total": 3 * gemm_fwd + attn_fwd_fl + attn_bwd_fl}
