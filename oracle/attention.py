"""Oracle causal multi-head / grouped-query attention, forward and backward.

Test infrastructure only (see ``oracle/__init__.py``).

What is followed:

* Sec. 4.1, Algorithm 1 (memory-resident Attention Backward): the backward
  pass produces the query gradient GQ and the key/value gradients GK, GV from
  the query tile, the output gradient GO, the softmax probabilities P and the
  key/value tiles, through GP = GO V^T, GS = SoftmaxBackward(P, GP),
  GV = P^T GO, GQ = GS K and GK = GS^T Q.
* The forward is not spelled out in the paper (it only says the backward
  reads the probabilities the forward produced); it is read as standard
  scaled-dot-product softmax attention of a decoder-only model.

Readings where the paper is silent (each is also listed in the design doc):

* scale: scores are ``scale * q . k`` with ``scale`` passed explicitly
  (1/sqrt(d) in every workload); GQ and GK carry the factor, GV does not.
* causal mask: query i sees keys j <= i (0-based, equal query/key lengths);
  masked probabilities are exactly 0.  No row is empty.
* SoftmaxBackward(P, GP) is the Jacobian-vector product of a row softmax:
  GS_ij = P_ij * (GP_ij - sum_k P_ik GP_ik).
* GQA: query head h reads key/value head floor(h / g), g = Hq / Hkv; the
  gradient of a key/value head sums over its g query heads.
* LSE is the natural-log row log-sum-exp of the (scaled, masked) scores.

Everything is float64.  The full S x S score matrix of one head is formed
explicitly (brute force, no online softmax, no tiling).
"""

import numpy as np


def _causal_mask(sq, sk):
    """Boolean [sq, sk] matrix, True where key j is visible to query i."""
    i = np.arange(sq)[:, None]
    j = np.arange(sk)[None, :]
    return j <= i


def attn_head_fwd(q, k, v, scale, causal=True):
    """One head.  q [Sq, D], k, v [Sk, D]  ->  (O [Sq, D], LSE [Sq], P [Sq, Sk])."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    s = float(scale) * (q @ k.T)                       # scores
    if causal:
        s = np.where(_causal_mask(q.shape[0], k.shape[0]), s, -np.inf)
    m = s.max(axis=1)                                  # row maximum (finite: key 0 always visible)
    e = np.exp(s - m[:, None])                         # exp(-inf) = 0 on masked entries
    l = e.sum(axis=1)
    p = e / l[:, None]                                 # softmax rows
    o = p @ v
    lse = m + np.log(l)
    return o, lse, p


def attn_head_bwd(q, k, v, do, scale, causal=True):
    """One head, gradient of sum(O * dO).

    Returns dict with dq [Sq, D], dk [Sk, D], dv [Sk, D] and the
    intermediates p, dp, delta (row term), ds.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    do = np.asarray(do, dtype=np.float64)
    _, _, p = attn_head_fwd(q, k, v, scale, causal)
    dp = do @ v.T                                      # GP = GO V^T
    delta = (p * dp).sum(axis=1)                       # sum_k P_ik GP_ik
    ds = p * (dp - delta[:, None])                     # GS = SoftmaxBackward(P, GP)
    dv = p.T @ do                                      # GV = P^T GO
    dq = float(scale) * (ds @ k)                       # GQ = GS K   (d s / d q = scale * k)
    dk = float(scale) * (ds.T @ q)                     # GK = GS^T Q
    return {"dq": dq, "dk": dk, "dv": dv, "p": p, "dp": dp, "delta": delta, "ds": ds}


def _check_shapes(q, k, v):
    if q.ndim != 4 or k.ndim != 4 or v.ndim != 4:
        raise ValueError("q, k, v must be [B, S, H, D]")
    B, S, Hq, D = q.shape
    if k.shape != v.shape or k.shape[0] != B or k.shape[1] != S or k.shape[3] != D:
        raise ValueError(f"shape mismatch q{q.shape} k{k.shape} v{v.shape}")
    Hkv = k.shape[2]
    if Hq % Hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    return B, S, Hq, Hkv, D


def attn_fwd(q, k, v, scale, causal=True, heads=None):
    """Batched forward.  q [B,S,Hq,D], k, v [B,S,Hkv,D].

    Returns O [B,S,Hq,D] and LSE [B,Hq,S] (float64).  ``heads`` optionally
    restricts the work to a list of (b, h) pairs; other entries are NaN.
    """
    B, S, Hq, Hkv, D = _check_shapes(q, k, v)
    g = Hq // Hkv
    o = np.full((B, S, Hq, D), np.nan)
    lse = np.full((B, Hq, S), np.nan)
    pairs = heads if heads is not None else [(b, h) for b in range(B) for h in range(Hq)]
    for b, h in pairs:
        kv = h // g
        o[b, :, h, :], lse[b, h, :], _ = attn_head_fwd(
            q[b, :, h, :], k[b, :, kv, :], v[b, :, kv, :], scale, causal)
    return o, lse


def attn_bwd(q, k, v, do, scale, causal=True, kv_heads=None):
    """Batched backward of sum(O * dO).

    Returns dq [B,S,Hq,D], dk, dv [B,S,Hkv,D] and delta [B,Hq,S] (float64).
    ``kv_heads`` optionally restricts the work to a list of (b, kv) pairs
    (all g query heads of each are done); other entries are NaN.
    """
    B, S, Hq, Hkv, D = _check_shapes(q, k, v)
    g = Hq // Hkv
    dq = np.full((B, S, Hq, D), np.nan)
    dk = np.full((B, S, Hkv, D), np.nan)
    dv = np.full((B, S, Hkv, D), np.nan)
    delta = np.full((B, Hq, S), np.nan)
    pairs = kv_heads if kv_heads is not None else [(b, kv) for b in range(B) for kv in range(Hkv)]
    for b, kv in pairs:
        dk_acc = np.zeros((S, D))
        dv_acc = np.zeros((S, D))
        for h in range(kv * g, kv * g + g):            # the g query heads sharing kv head `kv`
            r = attn_head_bwd(q[b, :, h, :], k[b, :, kv, :], v[b, :, kv, :],
                              do[b, :, h, :], scale, causal)
            dq[b, :, h, :] = r["dq"]
            delta[b, h, :] = r["delta"]
            dk_acc += r["dk"]
            dv_acc += r["dv"]
        dk[b, :, kv, :] = dk_acc
        dv[b, :, kv, :] = dv_acc
    return dq, dk, dv, delta
