"""Pins of the exponential parametrizations (oracle/expo.py):

X1  the exponential map against scipy.linalg.expm of the same normalized
    skew matrix, within the truncation bound |A|^(p+1) e^|A| / (p+1)!;
X2  2 x 2 rotations (closed form of the truncated sine and cosine series);
X3  orthogonality, det = +1, a symmetric W gives I;
X4  the explicit conv exponential against the implicit series of repeated
    circular convolutions (the theorem's two sides), the 1 x 1 kernel case
    against expm, skew-symmetry of conv(K - K*), orthogonality of the
    result through its Toeplitz singular values;
X5  planted mistakes.
"""

import math
import zlib

import numpy as np
import pytest
from scipy.linalg import expm

from oracle import conv, expo, spectral

RNG = np.random.default_rng(20260115)


@pytest.fixture(autouse=True)
def _rng_per_test(request):
    """Each test draws from a generator seeded by its own name, so that its
    inputs do not depend on which tests ran before it in the process (a
    parallel run deals tests to workers in any order)."""
    global RNG
    RNG = np.random.default_rng([20260115, zlib.crc32(request.node.name.encode())])


def trunc_bound(norm, p):
    return norm ** (p + 1) * math.exp(norm) / math.factorial(p + 1)


@pytest.mark.parametrize("c,p", [(8, 10), (32, 12), (64, 16), (5, 6)])
def test_exp_map_vs_expm(c, p):
    w = RNG.standard_normal((c, c))
    u = RNG.standard_normal(c)
    got, v = expo.exp_map(w, p, u, 3)
    a = w - w.T
    _, _, sigma, _ = spectral.spectral_prescale(a, u, 3)
    ahat = a / sigma
    nrm = np.linalg.norm(ahat, 2)
    ref = expm(ahat)
    assert np.max(np.abs(got - ref)) <= trunc_bound(nrm, p) + 1e-13
    assert np.max(np.abs(got.T @ got - np.eye(c))) <= 3 * trunc_bound(nrm, p) + 1e-12
    assert np.linalg.det(got) > 0


@pytest.mark.parametrize("a,p", [(2.0, 8), (-0.5, 9), (3.0, 20)])
def test_exp_map_rotation(a, p):
    w = np.array([[0.0, a], [0.0, 0.0]])
    got, _ = expo.exp_map(w, p, np.array([1.0, 0.0]), 1)
    sgn = 1.0 if a > 0 else -1.0
    cos_p = sum((-1) ** (k // 2) / math.factorial(k) for k in range(0, p + 1, 2))
    sin_p = sum((-1) ** ((k - 1) // 2) / math.factorial(k) for k in range(1, p + 1, 2))
    np.testing.assert_allclose(got, [[cos_p, sgn * sin_p], [-sgn * sin_p, cos_p]], rtol=0, atol=1e-15)


def test_exp_map_symmetric_is_identity():
    s = RNG.standard_normal((6, 6))
    got, v = expo.exp_map(s + s.T, 10, np.ones(6), 2)
    assert np.array_equal(got, np.eye(6)) and np.array_equal(v, np.ones(6))


def implicit_series(lk, x, p):
    """sum_j conv(L, .)^j x / j!: the per-input series the theorem replaces."""
    out = x.copy()
    term = x.copy()
    for j in range(1, p + 1):
        term = conv.conv_circular(lk, term) / j
        out = out + term
    return out


@pytest.mark.parametrize("c,k,p,scale,hw", [(4, 3, 4, 0.3, 8), (6, 3, 6, 0.2, 10), (3, 5, 3, 0.25, 12),
                                            (5, 3, 2, 1.0, 6)])
def test_conv_exp_explicit_equals_implicit(c, k, p, scale, hw):
    kern = RNG.standard_normal((c, c, k, k))
    e = expo.conv_exp(kern, p, scale)
    assert e.shape == (c, c, p * (k - 1) + 1, p * (k - 1) + 1)
    x = RNG.standard_normal((2, c, hw, hw))
    lk = scale * expo.skew_kernel(kern)
    np.testing.assert_allclose(conv.conv_circular(e, x), implicit_series(lk, x, p), rtol=0, atol=1e-11)


def test_conv_exp_1x1_is_matrix_exponential():
    kern = RNG.standard_normal((7, 7, 1, 1))
    e = expo.conv_exp(kern, 18, 0.3)
    l = 0.3 * (kern[:, :, 0, 0] - kern[:, :, 0, 0].T)
    assert np.max(np.abs(e[:, :, 0, 0] - expm(l))) <= trunc_bound(np.linalg.norm(l, 2), 18) + 1e-13


def test_skew_kernel_gives_skew_operator():
    kern = RNG.standard_normal((4, 4, 3, 3))
    lk = expo.skew_kernel(kern)
    x = RNG.standard_normal((1, 4, 6, 6))
    y = RNG.standard_normal((1, 4, 6, 6))
    lhs = np.sum(conv.conv_circular(lk, x) * y)
    rhs = -np.sum(x * conv.conv_circular(lk, y))
    assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(lhs))
    # and the adjoint kernel gives the adjoint operator
    adj = expo.adjoint_kernel(kern)
    assert abs(np.sum(conv.conv_circular(kern, x) * y) - np.sum(x * conv.conv_circular(adj, y))) <= 1e-11


def test_conv_exp_is_orthogonal():
    """With |conv(L)| small the truncated exponential is orthogonal up to the
    truncation bound: every Toeplitz singular value is within it of 1."""
    c, k, p, hw = 3, 3, 12, 6
    kern = RNG.standard_normal((c, c, k, k))
    lk = expo.skew_kernel(kern)
    nrm = np.linalg.svd(conv.toeplitz_matrix(lk, hw, hw), compute_uv=False)[0]
    scale = 0.8 / nrm
    e = expo.conv_exp(kern, p, scale)
    sv = conv.toeplitz_singular_values(e, hw, hw)
    assert np.max(np.abs(sv - 1.0)) <= 3 * trunc_bound(0.8, p) + 1e-12


def test_planted_unflipped_adjoint(monkeypatch):
    monkeypatch.setattr(expo, "adjoint_kernel", lambda k: np.transpose(np.asarray(k, float), (1, 0, 2, 3)).copy())
    with pytest.raises(AssertionError):
        test_skew_kernel_gives_skew_operator()


def test_planted_missing_factorial(monkeypatch):
    orig = expo.conv_exp

    def wrong(kern, terms, scale=1.0):
        # every power added without the 1/j! factor
        kern = np.asarray(kern, dtype=np.float64)
        c, _, k, _ = kern.shape
        lk = scale * expo.skew_kernel(kern)
        size = terms * (k - 1) + 1
        out = np.zeros((c, c, size, size))
        mid = (size - 1) // 2
        out[:, :, mid, mid] = np.eye(c)
        from oracle import aoc
        power = aoc.identity_kernel(c)
        for j in range(1, terms + 1):
            power = aoc.block_conv(power, lk)
            off = (size - power.shape[2]) // 2
            out[:, :, off:off + power.shape[2], off:off + power.shape[2]] += power
        return out
    monkeypatch.setattr(expo, "conv_exp", wrong)
    with pytest.raises(AssertionError):
        test_conv_exp_explicit_equals_implicit(4, 3, 4, 0.3, 8)
