"""Pins for the oracle GEMM (CPU only).

Each test fixes the oracle against something other than itself: a pure-Python
triple loop, exact integer arithmetic, closed forms, a hand-computed worked
example, and a planted mistake that the pins must catch.
"""

import itertools

import numpy as np
import pytest

from oracle import gemm, gemm_entries
from paper_2606_10415_amd.synth import normal_f16, uniform_int_f16
from conftest import load_golden


def _stored(x, trans):
    """Store logical matrix x in the layout that op(.) with `trans` expects."""
    return np.ascontiguousarray(x.T) if trans else x


def _brute(transA, transB, alpha, A, B, beta, C):
    """Pure-Python triple loop over Python floats (no numpy arithmetic)."""
    a = A.T.tolist() if transA else A.tolist()
    b = B.T.tolist() if transB else B.tolist()
    M, K, N = len(a), len(b), len(b[0])
    out = []
    for m in range(M):
        row = []
        for n in range(N):
            s = 0.0
            for k in range(K):
                s += float(a[m][k]) * float(b[k][n])
            v = alpha * s
            if beta != 0.0:
                v += beta * float(C[m][n])
            row.append(v)
        out.append(row)
    return np.array(out)


@pytest.mark.parametrize("transA,transB", list(itertools.product([0, 1], [0, 1])))
def test_gemm_matches_triple_loop(transA, transB):
    M, N, K = 5, 7, 9
    a = normal_f16(11, (M, K)).astype(np.float64)
    b = normal_f16(12, (K, N)).astype(np.float64)
    c = normal_f16(13, (M, N)).astype(np.float64)
    A, B = _stored(a, transA), _stored(b, transB)
    got = gemm(transA, transB, 0.75, A, B, -1.25, c)
    ref = _brute(transA, transB, 0.75, A, B, -1.25, c)
    np.testing.assert_allclose(got, ref, rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("transA,transB", list(itertools.product([0, 1], [0, 1])))
def test_gemm_exact_integers(transA, transB):
    # entries in {-2..2}, K = 1000: every partial sum is an integer, exact in float64.
    M, N, K = 6, 10, 1000
    a = uniform_int_f16(21, (M, K), -2, 2).astype(np.int64)
    b = uniform_int_f16(22, (K, N), -2, 2).astype(np.int64)
    c = uniform_int_f16(23, (M, N), -2, 2).astype(np.int64)
    exact = 3 * (a @ b) - 2 * c          # integer arithmetic
    A, B = _stored(a.astype(np.float16), transA), _stored(b.astype(np.float16), transB)
    got = gemm(transA, transB, 3.0, A, B, -2.0, c.astype(np.float16))
    assert np.array_equal(got, exact.astype(np.float64))


def test_gemm_closed_forms():
    M, N, K = 8, 6, 8
    b = normal_f16(31, (K, N))
    eye = np.eye(M, K, dtype=np.float16)
    assert np.array_equal(gemm(0, 0, 1.0, eye, b), b.astype(np.float64))
    ones_a = np.ones((M, K), np.float16)
    ones_b = np.ones((K, N), np.float16)
    assert np.array_equal(gemm(0, 0, 1.0, ones_a, ones_b), np.full((M, N), float(K)))
    # beta only: K = 0 is an empty sum
    c = normal_f16(32, (M, N))
    got = gemm(0, 0, 1.0, np.zeros((M, 0), np.float16), np.zeros((0, N), np.float16), 0.5, c)
    assert np.array_equal(got, 0.5 * c.astype(np.float64))


def test_gemm_transpose_consistency():
    M, N, K = 7, 5, 11
    a = normal_f16(41, (M, K))
    w = normal_f16(42, (N, K))          # nn.Linear weight layout [out, in]
    nt = gemm(0, 1, 1.0, a, w)
    nn = gemm(0, 0, 1.0, a, np.ascontiguousarray(w.T))
    tn = gemm(1, 0, 1.0, np.ascontiguousarray(a.T), np.ascontiguousarray(w.T))
    tt = gemm(1, 1, 1.0, np.ascontiguousarray(a.T), w)
    for x in (nn, tn, tt):
        np.testing.assert_array_equal(nt, x)


def test_gemm_beta_zero_never_reads_c():
    a = normal_f16(51, (4, 8))
    b = normal_f16(52, (8, 4))
    c = np.full((4, 4), np.nan, np.float16)
    assert np.isfinite(gemm(0, 0, 1.0, a, b, 0.0, c)).all()


def test_gemm_worked_example():
    g = load_golden("gemm_worked_example.json")
    A = np.array(g["A"], np.float16)
    B = np.array(g["B"], np.float16)
    C = np.array(g["C"], np.float16)
    assert np.array_equal(gemm(0, 0, 1.0, A, B), np.array(g["AB"], np.float64))
    assert np.array_equal(gemm(0, 0, g["alpha"], A, B, g["beta"], C), np.array(g["expected"], np.float64))
    At, Bt = np.ascontiguousarray(A.T), np.ascontiguousarray(B.T)
    assert np.array_equal(gemm(1, 1, g["alpha"], At, Bt, g["beta"], C), np.array(g["expected"], np.float64))


def test_gemm_entries_match_definition():
    M, N, K = 9, 13, 17
    for transA, transB in itertools.product([0, 1], [0, 1]):
        a = normal_f16(61, (M, K)).astype(np.float64)
        b = normal_f16(62, (K, N)).astype(np.float64)
        c = normal_f16(63, (M, N))
        A, B = _stored(a, transA), _stored(b, transB)
        rows = np.array([0, 3, 8, 8, 5])
        cols = np.array([12, 0, 4, 12, 7])
        got = gemm_entries(transA, transB, 1.5, A, B, 0.5, c, rows, cols)
        ref = _brute(transA, transB, 1.5, A, B, 0.5, c)[rows, cols]
        np.testing.assert_allclose(got, ref, rtol=1e-13, atol=1e-13)


def test_planted_transpose_mistake_is_caught():
    """A GEMM that ignores transB (a plausible layout slip) must fail the triple-loop pin."""
    def broken(transA, transB, alpha, A, B):
        a = np.asarray(A, np.float64)
        return alpha * ((a.T if transA else a) @ np.asarray(B, np.float64))
    a = normal_f16(71, (6, 6)).astype(np.float64)
    w = normal_f16(72, (6, 6)).astype(np.float64)
    ref = _brute(0, 1, 1.0, a, w, 0.0, None)
    assert not np.allclose(broken(0, 1, 1.0, a, w), ref)
    assert np.allclose(gemm(0, 1, 1.0, a, w), ref)
