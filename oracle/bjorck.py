"""Björck–Bowie orthogonalization, float64, written from Appendix A.5.

The paper defines the fixed-point iteration

    W_{t+1} = (1 + beta) W_t - beta W_t W_t^T W_t,      beta in (0, 1/2],

used with beta = 1/2 and a fixed number of iterations (12-25 "in practice").
The workloads pre-scale by the Frobenius norm, W_0 = W / ||W||_F, which puts
every singular value of W_0 in (0, 1] and therefore inside the basin of
convergence (0, sqrt(3)) of the scalar map f(x) = (1+beta) x - beta x^3.

The product W W^T W is evaluated through the smaller Gram matrix
(W (W^T W) when rows >= cols, (W W^T) W otherwise).  Both groupings are the
same matrix; the grouping only changes rounding.

Pins (tests/test_oracle_pins.py): P1 closed form through the SVD, P2
convergence, P3 orthogonal input, P4 scale invariance, and a hand-derived
golden value (tests/golden/bjorck_hand.json).
"""

import numpy as np

# Per-matrix status, mirroring what a caller is told about degenerate inputs.
STATUS_OK = 0
STATUS_ZERO = 1        # ||W||_F == 0: output is the zero matrix
STATUS_NONFINITE = 2   # a NaN or Inf in the input: output is all NaN


def frobenius_prescale(w):
    """Return (W / ||W||_F, status).  Float64 throughout."""
    w = np.asarray(w, dtype=np.float64)
    if not np.all(np.isfinite(w)):
        return np.full(w.shape, np.nan), STATUS_NONFINITE
    norm = np.sqrt(np.sum(w * w))
    if norm == 0.0:
        return np.zeros(w.shape), STATUS_ZERO
    return w / norm, STATUS_OK


def bjorck_step(w, beta=0.5):
    """One application of the Appendix A.5 update to a float64 matrix."""
    rows, cols = w.shape
    if rows >= cols:
        cubic = w @ (w.T @ w)
    else:
        cubic = (w @ w.T) @ w
    return (1.0 + beta) * w - beta * cubic


def bjorck(w, iters, beta=0.5, prescale="frobenius", return_status=False):
    """Orthogonalize one matrix: optional Frobenius pre-scaling, then exactly
    ``iters`` Björck steps (no early exit).

    ``prescale`` is "frobenius" or "none".  Rows >= cols gives orthonormal
    columns in the limit, rows < cols orthonormal rows.
    """
    if not (0.0 < beta <= 0.5):
        raise ValueError("beta must lie in (0, 1/2]")
    if iters < 0:
        raise ValueError("iters must be >= 0")
    w = np.asarray(w, dtype=np.float64)
    if prescale == "frobenius":
        w, status = frobenius_prescale(w)
    elif prescale == "none":
        status = STATUS_OK if np.all(np.isfinite(w)) else STATUS_NONFINITE
        if status != STATUS_OK:
            w = np.full(w.shape, np.nan)
    else:
        raise ValueError("prescale must be 'frobenius' or 'none'")
    if status == STATUS_OK:
        for _ in range(iters):
            w = bjorck_step(w, beta)
    if return_status:
        return w, status
    return w


def iterations_to_converge(w, tol=1e-5, beta=0.5, max_iters=200):
    """Smallest T with max_i |f^T(s_i)^2 - 1| <= tol, where s_i are the
    singular values of W / ||W||_F.  Used to choose iteration counts at
    which every matrix of a workload has converged."""
    w = np.asarray(w, dtype=np.float64)
    norm = np.sqrt(np.sum(w * w))
    s = np.linalg.svd(w, compute_uv=False) / norm
    for t in range(max_iters + 1):
        if np.max(np.abs(s * s - 1.0)) <= tol:
            return t
        s = (1.0 + beta) * s - beta * s ** 3
    return None
