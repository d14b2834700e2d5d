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


def spectral_prescale_vjp(w, u, power_iters, grad_w0):
    """dL/dW of W_0 = W / sigma(W) (spectral_prescale) given dL/dW_0, the
    cached vector u held constant (it is state carried between parameter
    steps, not a function of this step's W).

    With X the tall orientation, G_0 = dL/dX_0 and sigma = max(sigma_hat,
    ||X||_F / sqrt(N)):

        dL/dX = G_0 / sigma + c d(sigma)/dX,   c = -<G_0, X> / sigma^2.

    Frobenius branch (sigma_hat < ||X||_F / sqrt(N), ties go to sigma_hat
    as in the forward's max): d(sigma)/dX = X / (||X||_F sqrt(N)).
    Power-iteration branch: sigma_hat = |y| / |x| with x = X v, y = X^T x
    and v = v_{q-1} the vector before the last step; every earlier vector
    v_k = y_k / |y_k| depends on X as well, down to the constant v_0.  The
    chain rule through one step, written out with a = |y|, b = |x|:

        last step:  yh = c y / (a b),  gx = -c a x / b^3 + X yh,
                    dL/dX += x yh^T + gx v^T,   dL/dv = X^T gx;
        earlier:    gy = (dL/dv_k - <dL/dv_k, v_k> v_k) / |y_k|,
                    dL/dX += x_k gy^T + (X gy) v_{k-1}^T,
                    dL/dv_{k-1} = X^T X gy.

    Zero matrix: zero gradient; non-finite: all NaN (the forward's
    statuses)."""
    w = np.asarray(w, dtype=np.float64)
    rows, cols = w.shape
    n = min(rows, cols)
    g0 = np.asarray(grad_w0, dtype=np.float64)
    if not np.all(np.isfinite(w)):
        return np.full(w.shape, np.nan)
    fro = np.sqrt(np.sum(w * w))
    if fro == 0.0:
        return np.zeros(w.shape)
    tall = rows >= cols
    X = w if tall else w.T
    G = g0 if tall else g0.T
    u = np.asarray(u, dtype=np.float64).reshape(n)
    nv = np.sqrt(np.sum(u * u))
    v = u / nv if (nv > 0 and np.isfinite(nv)) else np.full(n, 1.0 / np.sqrt(n))
    # forward power iteration, keeping every vector
    vs, xs, ys = [v], [], []
    sigma_hat = 0.0
    for _ in range(power_iters):
        x = X @ vs[-1]
        y = X.T @ x
        ny = np.sqrt(np.sum(y * y))
        if ny == 0.0:
            sigma_hat = 0.0
            xs, ys = [], []
            break
        xs.append(x)
        ys.append(y)
        sigma_hat = ny / np.sqrt(np.sum(x * x))
        vs.append(y / ny)
    floor = fro / np.sqrt(n)
    sigma = max(sigma_hat, floor)
    c = -float(np.sum(G * X)) / sigma ** 2
    out = G / sigma
    if sigma_hat >= floor and xs:
        q = len(xs)
        x, y = xs[-1], ys[-1]
        a, b = np.sqrt(np.sum(y * y)), np.sqrt(np.sum(x * x))
        yh = c * y / (a * b)
        gx = -c * a * x / b ** 3 + X @ yh
        out = out + np.outer(x, yh) + np.outer(gx, vs[q - 1])
        gv = X.T @ gx
        for k in range(q - 1, 0, -1):           # v_k = y_k / |y_k| (step k, 1-based)
            yk, vk = ys[k - 1], vs[k]
            gy = (gv - np.sum(gv * vk) * vk) / np.sqrt(np.sum(yk * yk))
            xg = X @ gy
            out = out + np.outer(xs[k - 1], gy) + np.outer(xg, vs[k - 1])
            gv = X.T @ xg
    else:
        out = out + c * X / (fro * np.sqrt(n))
    return out if tall else out.T


def bjorck_spectral_vjp(w, u, grad_out, iters, power_iters=1, beta=0.5):
    """dL/dW for L depending on W through bjorck_spectral(W, u, iters,
    power_iters, beta)[0], given dL/d(output) = grad_out, u constant."""
    from . import bjorck_grad as _bg
    w0, _, _, status = spectral_prescale(w, u, power_iters)
    if status == _bj.STATUS_NONFINITE:
        return np.full(np.shape(w), np.nan)
    if status == _bj.STATUS_ZERO:
        return np.zeros(np.shape(w))
    g0 = _bg.bjorck_vjp(w0, grad_out, iters, beta, prescale="none")
    return spectral_prescale_vjp(w, u, power_iters, g0)
