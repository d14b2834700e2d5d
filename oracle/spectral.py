"""Spectral pre-scaling by power iteration with a caller-owned cached
vector, float64 (Appendix A.5: spectral normalization of W_0 before the
Björck iteration, reusing a cached power-iteration estimate of the top
singular vector across updates; Section 2: spectral normalization by batched
power iteration).

Reading (the paper gives no formulas for this step): with X the tall
orientation of W (X = W if rows >= cols, else W^T; N = min(rows, cols)) and
v the cached vector of length N (a right singular vector estimate of X),

    v <- v / ||v||            (a zero vector is replaced by ones / sqrt(N))
    repeat q >= 1 times:
        x = X v,  y = X^T x
        if ||y|| == 0: stop   (sigma_hat = 0)
        sigma_hat = ||y|| / ||x||,  v <- y / ||y||
    sigma = max(sigma_hat, ||W||_F / sqrt(N))
    W_0 = W / sigma,  and v is handed back as the new cache.

||X^T X v|| / ||X v|| for a unit v lies between ||X v|| and sigma_max, and
||W||_F / sqrt(N) <= sigma_max too, so sigma never exceeds sigma_max and the
largest singular value of W_0 is at least 1.  The second bound replaces a
useless estimate (a cached vector in or near the null space of W).  The
iteration converges when sigma_max / sigma < sqrt(3) (the basin of the scalar
map); a cached vector from the previous parameter step gives sigma within a
fraction of a percent of sigma_max, a random start with one step about
sigma_max / sqrt(2) on square Gaussian matrices.  Zero and non-finite
matrices get the statuses of the Frobenius path and leave the vector
unchanged.

Pins (tests/test_oracle_spectral_pins.py): hand-computed diagonal cases
(tests/golden/spectral_hand.json), convergence to the SVD's top singular
pair, the bounds above on random matrices, the transpose relation, and the
saving in Björck iterations that motivates the step, and a planted missing
lower bound.
"""

import numpy as np

from . import bjorck as _bj


def spectral_prescale(w, u, power_iters):
    """Return (W_0, new vector, sigma, status)."""
    if power_iters < 1:
        raise ValueError("power_iters must be >= 1")
    w = np.asarray(w, dtype=np.float64)
    rows, cols = w.shape
    n = min(rows, cols)
    u = np.asarray(u, dtype=np.float64).reshape(n)
    if not np.all(np.isfinite(w)):
        return np.full(w.shape, np.nan), u.copy(), np.nan, _bj.STATUS_NONFINITE
    fro = np.sqrt(np.sum(w * w))
    if fro == 0.0:
        return np.zeros(w.shape), u.copy(), 0.0, _bj.STATUS_ZERO
    x_mat = w if rows >= cols else w.T
    nv = np.sqrt(np.sum(u * u))
    v = u / nv if (nv > 0 and np.isfinite(nv)) else np.full(n, 1.0 / np.sqrt(n))
    sigma_hat = 0.0
    for _ in range(power_iters):
        x = x_mat @ v
        y = x_mat.T @ x
        ny = np.sqrt(np.sum(y * y))
        if ny == 0.0:
            sigma_hat = 0.0
            break
        sigma_hat = ny / np.sqrt(np.sum(x * x))
        v = y / ny
    sigma = max(sigma_hat, fro / np.sqrt(n))
    return w / sigma, v, sigma, _bj.STATUS_OK


def bjorck_spectral(w, u, iters, power_iters=1, beta=0.5):
    """Spectral pre-scaling, then exactly ``iters`` Björck steps.
    Returns (output, new vector, status)."""
    w0, v, _, status = spectral_prescale(w, u, power_iters)
    if status == _bj.STATUS_OK:
        for _ in range(iters):
            w0 = _bj.bjorck_step(w0, beta)
    return w0, v, status


def iterations_to_converge_scaled(w, scale, tol=1e-5, beta=0.5, max_iters=400):
    """Smallest T with max_i |f^T(s_i)^2 - 1| <= tol for the singular values
    s_i of W / scale (the scalar map of the iteration, as in
    bjorck.iterations_to_converge)."""
    s = np.linalg.svd(np.asarray(w, dtype=np.float64), compute_uv=False) / scale
    for t in range(max_iters + 1):
        if np.max(np.abs(s * s - 1.0)) <= tol:
            return t
        s = (1.0 + beta) * s - beta * s ** 3
    return None
