"""Matrices W = Q D with Q the first n columns of a Householder reflection
H = I - 2 v v^T (orthonormal columns) and D = diag(d), built in
O(rows x cols) time and memory for any size.  The Bjorck iteration keeps
the Q factor (X = Q Y gives X^T X = Y^T Y and X X^T X = Q Y Y^T Y, so
every step maps Q Y_t to Q Y_{t+1}, and ||Q D||_F = ||D||_F for the
pre-scaling), hence Bjorck(Q D) = Q Bjorck(D): the reference of a huge
matrix is the oracle's iteration on the n x n diagonal D, lifted by Q
(`lift`).  test_oracle_pins.py pins this against the oracle run on the
dense Q D."""

import numpy as np


def factors(seed, rows, cols, lo=0.4, hi=1.0):
    """(v, d): a unit vector v of length max(rows, cols) and n = min(rows,
    cols) diagonal values in [lo, hi], from a seeded generator."""
    rng = np.random.default_rng(seed)
    m, n = max(rows, cols), min(rows, cols)
    v = rng.standard_normal(m)
    v /= np.linalg.norm(v)
    return v, rng.uniform(lo, hi, n)


def lift(v, y):
    """Q y for Q = (I - 2 v v^T)[:, :n] and an n x n matrix y, as
    [y; 0] - 2 v (y^T v[:n])^T."""
    n = y.shape[0]
    out = -2.0 * np.outer(v, y.T @ v[:n])
    out[:n] += y
    return out


def matrix(v, d, rows, cols):
    """W = Q diag(d) in float64, in the requested orientation (a wide
    shape is the transpose of the tall one)."""
    w = lift(v, np.diag(d))
    return w if rows >= cols else w.T
