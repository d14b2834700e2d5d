"""Exponential parametrizations, float64: the exponential map of a
skew-symmetric matrix with spectral normalization (Appendix A.3, algorithm
"Exponential Map with Spectral Normalization") and the explicit exponential
of a skew-symmetric convolution kernel by the block-convolution operator
(Appendix B.2, theorem "Explicit conv exponential", Adaptive-SOC).

Exponential map (square C x C parameter W, p terms):
    A = W - W^T,  Ahat = A / ||A||_2,  What = sum_{k=0}^{p} Ahat^k / k!
computed with the algorithm's recurrence P_0 = I, P_k = P_{k-1} Ahat / k,
What = sum_k P_k.  ||A||_2 is read as the spectral-normalization estimate
of oracle/spectral.py (power iteration from a cached vector, with the lower
bound ||A||_F / sqrt(C)); a zero A gives What = I.

Conv exponential (square kernel K of c x c x k x k, odd k, stride 1):
    L = K - K*,  K*[o, i, a, b] = K[i, o, k-1-a, k-1-b]   (the kernel of the
                                                           adjoint conv)
    E = sum_{j=0}^{p} L^(⊛j) / j!
with L^(⊛0) the 1x1 identity and L^(⊛j) of size j (k-1) + 1; terms are
summed centred in the final (p (k-1) + 1)^2 grid, which keeps
conv(E, x) = sum_j conv(L, .)^j x / j! for centred ("same") circular
padding.  An optional scale t multiplies L first (exp(t L)).

Pins (tests/test_oracle_expo_pins.py): scipy.linalg.expm within the
truncation bound, 2 x 2 rotations, orthogonality and det = +1, the implicit
series of repeated convolutions against the explicit kernel, skew-symmetry
of conv(L), the 1 x 1 kernel case against expm.
"""

import math

import numpy as np

from . import aoc as _aoc
from . import spectral as _sp


def exp_map(w, terms, u, power_iters=1):
    """Returns (What, new cached vector)."""
    w = np.asarray(w, dtype=np.float64)
    if w.shape[0] != w.shape[1]:
        raise ValueError("the exponential map needs a square matrix")
    a = w - w.T
    c = w.shape[0]
    _, v, sigma, status = _sp.spectral_prescale(a, u, power_iters)
    if status == 1:          # A == 0: exp(0) = I, the vector is left as it was
        return np.eye(c), np.asarray(u, dtype=np.float64).copy()
    if status == 2:
        return np.full((c, c), np.nan), np.asarray(u, dtype=np.float64).copy()
    ahat = a / sigma
    out = np.eye(c)
    p = np.eye(c)
    for k in range(1, terms + 1):
        p = p @ ahat / k
        out = out + p
    return out, v


def adjoint_kernel(kern):
    """K*[o, i, a, b] = K[i, o, k-1-a, k-1-b]: the kernel whose circular
    convolution is the adjoint of conv(K, .) for stride 1 and centred
    padding (odd k)."""
    kern = np.asarray(kern, dtype=np.float64)
    return np.flip(np.transpose(kern, (1, 0, 2, 3)), axis=(2, 3)).copy()


def skew_kernel(kern):
    return np.asarray(kern, dtype=np.float64) - adjoint_kernel(kern)


def conv_exp(kern, terms, scale=1.0):
    """Explicit kernel of exp(scale * conv(K - K*)), p = terms."""
    kern = np.asarray(kern, dtype=np.float64)
    c, c2, k, k2 = kern.shape
    if c != c2 or k != k2 or k % 2 == 0:
        raise ValueError("square kernels with equal channels and odd size only")
    lk = scale * skew_kernel(kern)
    size = terms * (k - 1) + 1
    out = np.zeros((c, c, size, size))
    mid = (size - 1) // 2
    out[:, :, mid, mid] = np.eye(c)
    power = _aoc.identity_kernel(c)
    for j in range(1, terms + 1):
        power = _aoc.block_conv(power, lk) / j
        s = power.shape[2]
        off = (size - s) // 2
        out[:, :, off:off + s, off:off + s] += power
    return out
