"""Oracle GEMM (test infrastructure only; see ``oracle/__init__.py``).

Definition followed: Sec. 4.1, "FP16 GEMM assembly pipeline".  The backend
computes the GEMM primitives of the QKV, output and FFN projections and of the
attention-backward matmuls; the output tile C is loaded as the accumulation
buffer, so the primitive is an update C <- alpha * op(A) op(B) + beta * C.

Layout convention (row-major, as numpy/PyTorch store matrices):
    op(X) = X      if trans == 0
    op(X) = X^T    if trans == 1
A is stored [M, K] (trans 0) or [K, M] (trans 1); B is stored [K, N]
(trans 0) or [N, K] (trans 1); C is [M, N].

Everything is evaluated in float64 from the float16 input values.  beta == 0
never reads C (so NaN / garbage in C does not propagate), matching the
reading that beta scales an accumulation buffer that may be uninitialised.
"""

import numpy as np


def _op(x, trans):
    x = np.asarray(x, dtype=np.float64)
    return x.T if trans else x


def gemm(transA, transB, alpha, A, B, beta=0.0, C=None):
    """Return alpha * op(A) @ op(B) + beta * C as a float64 [M, N] array."""
    a = _op(A, transA)
    b = _op(B, transB)
    if a.shape[1] != b.shape[0]:
        raise ValueError(f"inner dims differ: {a.shape} x {b.shape}")
    out = float(alpha) * (a @ b)
    if beta != 0.0:
        if C is None:
            raise ValueError("beta != 0 needs C")
        out = out + float(beta) * np.asarray(C, dtype=np.float64)
    return out


def gemm_entries(transA, transB, alpha, A, B, beta, C, rows, cols):
    """Selected entries out[t] = (alpha*op(A)@op(B) + beta*C)[rows[t], cols[t]].

    Each entry is one float64 dot product of length K; used to check full-size
    GPU outputs at sampled positions without forming the whole product.
    """
    rows = np.asarray(rows, dtype=np.int64)
    cols = np.asarray(cols, dtype=np.int64)
    a = _op(A, transA)
    b = _op(B, transB)
    arow = np.asarray(a[rows, :], dtype=np.float64)      # [n, K]
    bcol = np.asarray(b[:, cols], dtype=np.float64).T    # [n, K]
    out = float(alpha) * np.einsum("nk,nk->n", arow, bcol)
    if beta != 0.0:
        out = out + float(beta) * np.asarray(C, dtype=np.float64)[rows, cols]
    return out


def column_sum(X):
    """Sum over the rows of X [T, N] in float64: the gradient of a bias that is
    broadcast over the T rows of a linear layer's output."""
    return np.sum(np.asarray(X, dtype=np.float64), axis=0)
