"""Pins of the oracle's RMSNorm and rotary embedding (CPU).

RMSNorm: central finite differences of sum(y * g) w.r.t. x and w; scale
invariance; the constant-row closed form; the orthogonality of dx to x that
scale invariance implies; a hand-derived worked example.
Rotary embedding: position 0 is the identity; every (i, i + d/2) pair keeps
its norm; scores depend only on the position difference; the backward is the
inverse rotation and matches finite differences; a hand-derived worked
example fixes the pairing and the signs.
Full layer (RMSNorm + rotary embedding + attention + SwiGLU MLP, with the
Qwen2.5 QKV bias): finite differences w.r.t. X, the four projection weights,
both RMSNorm weights and the QKV bias; with a zero QKV weight the attention
output equals the V bias (attention averages identical values); with Q and K
from the bias alone, the first off-diagonal score is the one the rotation of
the biased Q at position 1 gives, which fixes the bias before the rotation.
Column sum (the bias gradient): brute force over a small matrix.
"""

import numpy as np
import pytest

from conftest import golden_value, load_golden, rel_f
from oracle import (LayerNorms, LayerShape, column_sum, layer_bwd, layer_fwd, rmsnorm_bwd,
                    rmsnorm_fwd, rope_angles, rope_bwd, rope_fwd)


def _fd_grad(f, x, h=1e-6):
    g = np.zeros_like(x)
    it = np.nditer(x, flags=["multi_index"])
    for _ in it:
        i = it.multi_index
        xp = x.copy(); xp[i] += h
        xm = x.copy(); xm[i] -= h
        g[i] = (f(xp) - f(xm)) / (2 * h)
    return g


def test_rmsnorm_worked_example():
    gold = load_golden("rmsnorm_worked_example.json")
    x = np.array([[golden_value(v) for v in gold["x"]]])
    w = np.array([golden_value(v) for v in gold["w"]])
    dy = np.array([[golden_value(v) for v in gold["dy"]]])
    exp = gold["expected"]
    y, rstd = rmsnorm_fwd(x, w, 0.0)
    dx, dw = rmsnorm_bwd(dy, x, w, 0.0)
    np.testing.assert_allclose(rstd[0], golden_value(exp["rstd"]), rtol=1e-14)
    np.testing.assert_allclose(y[0], [golden_value(v) for v in exp["y"]], rtol=1e-14)
    np.testing.assert_allclose(dx[0], [golden_value(v) for v in exp["dx"]], rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(dw, [golden_value(v) for v in exp["dw"]], rtol=1e-14, atol=1e-15)


def test_rmsnorm_finite_differences():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((3, 8))
    w = rng.standard_normal(8)
    g = rng.standard_normal((3, 8))
    eps = 1e-3
    dx, dw = rmsnorm_bwd(g, x, w, eps)
    fx = _fd_grad(lambda xx: np.sum(rmsnorm_fwd(xx, w, eps)[0] * g), x)
    fw = _fd_grad(lambda ww: np.sum(rmsnorm_fwd(x, ww, eps)[0] * g), w)
    assert rel_f(dx, fx) <= 1e-6
    assert rel_f(dw, fw) <= 1e-6


def test_rmsnorm_scale_invariance_and_closed_form():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((4, 16))
    w = rng.standard_normal(16)
    y1, _ = rmsnorm_fwd(x, w, 0.0)
    y2, _ = rmsnorm_fwd(7.5 * x, w, 0.0)
    np.testing.assert_allclose(y1, y2, rtol=1e-13)
    # a constant row c: r = 1/|c|, y = sign(c) w
    c = np.full((2, 16), -2.5)
    y, r = rmsnorm_fwd(c, w, 0.0)
    np.testing.assert_allclose(r, 0.4, rtol=1e-14)
    np.testing.assert_allclose(y, -np.broadcast_to(w, (2, 16)), rtol=1e-14)
    # unit mean square of the normalised row
    np.testing.assert_allclose(np.mean((y1 / w) ** 2, axis=1), 1.0, rtol=1e-12)


def test_rmsnorm_gradient_orthogonal_to_input():
    """Scale invariance (eps = 0): d/da L(a x) = 0, i.e. sum_j dx_j x_j = 0 per row."""
    rng = np.random.default_rng(5)
    x = rng.standard_normal((5, 32))
    w = rng.standard_normal(32)
    g = rng.standard_normal((5, 32))
    dx, _ = rmsnorm_bwd(g, x, w, 0.0)
    assert np.max(np.abs(np.sum(dx * x, axis=1))) <= 1e-12 * np.max(np.abs(dx)) * 32


def test_rope_worked_example():
    gold = load_golden("rope_worked_example.json")
    base = golden_value(gold["base"])
    row = np.array([golden_value(v) for v in gold["x"]])
    x = np.stack([row, row])[None, :, None, :]          # [B=1, S=2, heads=1, D=4]
    y = rope_fwd(x, base)
    np.testing.assert_allclose(y[0, 0, 0], row, rtol=0, atol=0)
    np.testing.assert_allclose(y[0, 1, 0], [golden_value(v) for v in gold["expected"]["y_pos1"]],
                               rtol=1e-14)
    dy = np.zeros_like(x)
    dy[0, 1, 0, 0] = 1.0
    dx = rope_bwd(dy, base)
    np.testing.assert_allclose(dx[0, 1, 0], [golden_value(v) for v in gold["expected"]["dx_pos1_for_dy_e0"]],
                               rtol=1e-14, atol=1e-16)
    np.testing.assert_allclose(dx[0, 0, 0], 0.0, atol=0)


def test_rope_pair_norms_and_relative_positions():
    rng = np.random.default_rng(6)
    B, S, Hh, D = 2, 11, 3, 8
    x = rng.standard_normal((B, S, Hh, D))
    y = rope_fwd(x, 10000.0)
    h = D // 2
    np.testing.assert_allclose(x[..., :h] ** 2 + x[..., h:] ** 2, y[..., :h] ** 2 + y[..., h:] ** 2,
                               rtol=1e-12)
    # q at position p1, k at position p2: the rotated dot product depends on p1 - p2 only
    q = rng.standard_normal(D)
    k = rng.standard_normal(D)
    def rot(v, p):
        seq = np.zeros((1, p + 1, 1, D)); seq[0, p, 0] = v
        return rope_fwd(seq, 500.0)[0, p, 0]
    d1 = rot(q, 7) @ rot(k, 3)
    d2 = rot(q, 9) @ rot(k, 5)
    d3 = rot(q, 4) @ rot(k, 0)
    np.testing.assert_allclose([d2, d3], [d1, d1], rtol=1e-12)
    assert abs(rot(q, 7) @ rot(k, 7) - q @ k) <= 1e-12 * np.linalg.norm(q) * np.linalg.norm(k)


def test_rope_backward_is_inverse_and_matches_fd():
    rng = np.random.default_rng(7)
    x = rng.standard_normal((1, 5, 2, 6))
    g = rng.standard_normal((1, 5, 2, 6))
    np.testing.assert_allclose(rope_bwd(rope_fwd(x, 100.0), 100.0), x, rtol=1e-12, atol=1e-14)
    fd = _fd_grad(lambda xx: np.sum(rope_fwd(xx, 100.0) * g), x)
    assert rel_f(rope_bwd(g, 100.0), fd) <= 1e-8


def test_rope_angles_definition_points():
    a = rope_angles(3, 8, 10000.0)
    np.testing.assert_allclose(a[0], 0.0, atol=0)
    np.testing.assert_allclose(a[1, 0], 1.0, rtol=0)            # theta_0 = base^0
    np.testing.assert_allclose(a[2, 2], 2 * 10000.0 ** -0.5, rtol=1e-15)   # theta_2 = base^(-4/8)


SHAPE = LayerShape(B=2, S=5, H=16, Hq=4, Hkv=2, D=4, F=12)


def _full_params(seed):
    rng = np.random.default_rng(seed)
    sh = SHAPE
    p = {"X": rng.standard_normal((sh.T, sh.H)),
         "Wqkv": 0.3 * rng.standard_normal((sh.qkv_cols, sh.H)),
         "Wo": 0.3 * rng.standard_normal((sh.H, sh.Hq * sh.D)),
         "Wgu": 0.3 * rng.standard_normal((2 * sh.F, sh.H)),
         "Wd": 0.3 * rng.standard_normal((sh.H, sh.F)),
         "dY": rng.standard_normal((sh.T, sh.H))}
    norms = LayerNorms(wn1=1 + 0.2 * rng.standard_normal(sh.H), wn2=1 + 0.2 * rng.standard_normal(sh.H),
                       eps=1e-5, rope_base=50.0, bqkv=0.5 * rng.standard_normal(sh.qkv_cols))
    return p, norms


@pytest.mark.parametrize("which", ["X", "Wqkv", "Wo", "Wgu", "Wd", "wn1", "wn2", "bqkv"])
def test_full_layer_finite_differences(which):
    p, norms = _full_params(8)

    def loss(val):
        q = dict(p)
        n = norms
        if which in ("wn1", "wn2", "bqkv"):
            n = LayerNorms(**{**norms.__dict__, which: val})
        else:
            q[which] = val
        Y = layer_fwd(SHAPE, q["X"], q["Wqkv"], q["Wo"], q["Wgu"], q["Wd"], norm=n)["Y"]
        return float(np.sum(Y * p["dY"]))

    g = layer_bwd(SHAPE, p["X"], p["Wqkv"], p["Wo"], p["Wgu"], p["Wd"], p["dY"], norm=norms)
    key = {"X": "dX", "Wqkv": "dWqkv", "Wo": "dWo", "Wgu": "dWgu", "Wd": "dWd",
           "wn1": "dWn1", "wn2": "dWn2", "bqkv": "dbqkv"}[which]
    start = getattr(norms, which) if which in ("wn1", "wn2", "bqkv") else p[which]
    fd = _fd_grad(loss, np.array(start, dtype=np.float64))
    assert rel_f(g[key], fd) <= 1e-6


def test_planted_rope_sign_mistake_fails_fd():
    """A rotation with the wrong sign in the backward (a plausible slip) fails the layer FD."""
    import oracle.layer as L
    p, norms = _full_params(9)
    saved = L.rope_bwd
    try:
        L.rope_bwd = lambda dy, base: rope_fwd(dy, base)          # forward rotation instead of inverse
        g = layer_bwd(SHAPE, p["X"], p["Wqkv"], p["Wo"], p["Wgu"], p["Wd"], p["dY"], norm=norms)
    finally:
        L.rope_bwd = saved

    def loss(x):
        return float(np.sum(layer_fwd(SHAPE, x, p["Wqkv"], p["Wo"], p["Wgu"], p["Wd"], norm=norms)["Y"] * p["dY"]))
    fd = _fd_grad(loss, p["X"].copy())
    assert rel_f(g["dX"], fd) > 1e-3


def test_column_sum_brute_force():
    x = np.arange(12, dtype=np.float64).reshape(4, 3) - 5.5
    want = [sum(x[r][c] for r in range(4)) for c in range(3)]
    assert np.array_equal(column_sum(x), np.array(want))
    assert column_sum(np.zeros((0, 3))).tolist() == [0.0, 0.0, 0.0]


def test_qkv_bias_only_v_gives_v_bias():
    """Wqkv = 0 and a bias on the V columns only: every row of every head's
    attention output is its kv head's V bias (GQA: query head h reads kv head
    h // (Hq / Hkv)), whatever the scores."""
    p, norms = _full_params(10)
    sh = SHAPE
    b = np.zeros(sh.qkv_cols)
    bv = np.arange(sh.Hkv * sh.D, dtype=np.float64) * 0.25 - 1.0
    b[(sh.Hq + sh.Hkv) * sh.D:] = bv
    n = LayerNorms(**{**norms.__dict__, "bqkv": b})
    O = layer_fwd(sh, p["X"], np.zeros_like(p["Wqkv"]), p["Wo"], p["Wgu"], p["Wd"], norm=n)["O"]
    g = sh.Hq // sh.Hkv
    want = np.concatenate([bv[(h // g) * sh.D:(h // g + 1) * sh.D] for h in range(sh.Hq)])
    assert np.allclose(O, np.broadcast_to(want, O.shape), rtol=0, atol=1e-12)


def test_qkv_bias_is_added_before_the_rotation():
    """Wqkv = 0, Q and K from the bias alone.  Query 1 against key 0 scores
    (R_1 bq) . bk (the key at position 0 is unrotated); against key 1 the
    common rotation cancels and the score is bq . bk.  A bias added after the
    rotation would give bq . bk for both (LSE = log 2 + that score)."""
    p, norms = _full_params(11)
    sh = SHAPE
    rng = np.random.default_rng(12)
    bq = rng.standard_normal(sh.D)
    bk = rng.standard_normal(sh.D)
    b = np.zeros(sh.qkv_cols)
    b[:sh.Hq * sh.D] = np.tile(bq, sh.Hq)
    b[sh.Hq * sh.D:(sh.Hq + sh.Hkv) * sh.D] = np.tile(bk, sh.Hkv)
    n = LayerNorms(**{**norms.__dict__, "bqkv": b})
    lse = layer_fwd(sh, p["X"], np.zeros_like(p["Wqkv"]), p["Wo"], p["Wgu"], p["Wd"], norm=n)["LSE"]
    scale = 1.0 / np.sqrt(sh.D)
    q_at_1 = rope_fwd(np.stack([bq, bq])[None, :, None, :], norms.rope_base)[0, 1, 0]
    s10, s11 = scale * float(q_at_1 @ bk), scale * float(bq @ bk)
    assert abs(lse[0, 0, 1] - np.logaddexp(s10, s11)) <= 1e-12
    assert abs(lse[0, 0, 0] - s11) <= 1e-12
    assert abs(lse[0, 0, 1] - (np.log(2.0) + s11)) > 1e-3
