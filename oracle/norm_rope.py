"""Oracle RMSNorm and rotary position embedding (test infrastructure only).

The paper's text defines neither: it names the evaluated models (LLaMA-2,
Baichuan2, Qwen2.5; Sec. 6.1), whose decoder layers normalise the input of
the attention and FFN blocks with RMSNorm and rotate queries and keys with
rotary position embeddings.  Both are implemented here from their published
definitions, in float64:

* RMSNorm (Zhang & Sennrich, 2019), per token row x of width H:
      r = (mean_j x_j^2 + eps)^(-1/2),   y_j = w_j * x_j * r.
  Gradient of L with dL/dy = g:
      dx_j = r * w_j * g_j - r^3 * x_j / H * sum_i g_i * w_i * x_i,
      dw_j = sum over rows of g_j * x_j * r.
* Rotary embedding (Su et al., RoFormer, 2021), "rotate-half" pairing used by
  the LLaMA-2 and Qwen2.5 checkpoints: for head dimension d, frequency index
  i < d/2 and position p (0-based within the sequence),
      theta_i = base^(-2i/d),  a = p * theta_i,
      y_i       = x_i cos a - x_{i+d/2} sin a,
      y_{i+d/2} = x_{i+d/2} cos a + x_i sin a.
  The map is a rotation, so its gradient is the inverse rotation (angle -a).
"""

import numpy as np


def rmsnorm_fwd(x, w, eps):
    """x [T, H], w [H] -> (y [T, H], rstd [T]), float64."""
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    rstd = 1.0 / np.sqrt(np.mean(x * x, axis=1) + eps)
    return w * x * rstd[:, None], rstd


def rmsnorm_bwd(dy, x, w, eps):
    """Gradients of sum(y * dy) for y = rmsnorm_fwd(x, w, eps): (dx [T, H], dw [H])."""
    dy = np.asarray(dy, dtype=np.float64)
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    H = x.shape[1]
    rstd = 1.0 / np.sqrt(np.mean(x * x, axis=1) + eps)
    gw = dy * w
    dot = np.sum(gw * x, axis=1)
    dx = rstd[:, None] * gw - (rstd ** 3 * dot / H)[:, None] * x
    dw = np.sum(dy * x * rstd[:, None], axis=0)
    return dx, dw


def rope_angles(S, D, base):
    """a[p, i] = p * base^(-2i/D) for positions p < S and i < D/2, float64."""
    i = np.arange(D // 2, dtype=np.float64)
    theta = base ** (-2.0 * i / D)
    return np.arange(S, dtype=np.float64)[:, None] * theta[None, :]


def _rotate(x, angles, sign):
    """Rotate pairs (i, i + D/2) of x [B, S, heads, D] by sign * angles [S, D/2]."""
    x = np.asarray(x, dtype=np.float64)
    D = x.shape[-1]
    h = D // 2
    c = np.cos(angles)[None, :, None, :]
    s = sign * np.sin(angles)[None, :, None, :]
    x1, x2 = x[..., :h], x[..., h:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def rope_fwd(x, base):
    """Rotary embedding of x [B, S, heads, D] (positions 0..S-1 in every batch row)."""
    x = np.asarray(x, dtype=np.float64)
    return _rotate(x, rope_angles(x.shape[1], x.shape[3], base), 1.0)


def rope_bwd(dy, base):
    """Gradient of sum(rope_fwd(x) * dy) w.r.t. x: the inverse rotation of dy."""
    dy = np.asarray(dy, dtype=np.float64)
    return _rotate(dy, rope_angles(dy.shape[1], dy.shape[3], base), -1.0)
