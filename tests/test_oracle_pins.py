"""Pins of the CPU oracle against things other than itself: hand-derived
values, closed forms, invariants, textbook routines (numpy SVD, torch CPU
conv2d) and brute force.  Every test here runs on the CPU."""

import json
import math
import os
from decimal import Decimal

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import aoc, bjorck, checks, conv

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rand(rng, m, n):
    return rng.standard_normal((m, n)) / math.sqrt(n)


# ---------------------------------------------------------------- Björck ---

def test_golden_hand_values():
    with open(os.path.join(GOLDEN, "bjorck_hand.json")) as f:
        cases = json.load(f)["cases"]
    for case in cases:
        got = bjorck.bjorck(np.array(case["input"], dtype=np.float64), case["iters"])
        want = np.array([[float(Decimal(v)) for v in row] for row in case["expected"]])
        np.testing.assert_allclose(got, want, rtol=0, atol=1e-15, err_msg=case["name"])


@pytest.mark.parametrize("shape", [(16, 16), (16, 8), (8, 16), (64, 32), (33, 50), (1, 5), (7, 1)])
@pytest.mark.parametrize("beta", [0.5, 0.3])
def test_p1_closed_form_through_svd(shape, beta):
    """P1: the iteration acts on each singular value independently:
    W_T = U diag(f^T(s_i / ||W||_F)) V^T."""
    rng = np.random.default_rng(11)
    w = rand(rng, *shape)
    iters = 9
    u, s, vt = np.linalg.svd(w, full_matrices=False)
    x = s / np.sqrt(np.sum(s * s))
    for _ in range(iters):
        x = (1 + beta) * x - beta * x ** 3
    want = (u * x) @ vt
    got = bjorck.bjorck(w, iters, beta)
    assert checks.relative_difference(got, want) <= 1e-10


@pytest.mark.parametrize("shape,iters", [((16, 8), 12), ((64, 32), 15), ((256, 128), 15),
                                         ((40, 100), 20)])
def test_p2_rectangular_converges(shape, iters):
    """P2: rectangular Gaussian matrices converge at the workloads' T."""
    rng = np.random.default_rng(3)
    w = rand(rng, *shape)
    assert bjorck.iterations_to_converge(w) <= iters
    assert checks.gram_deviation(bjorck.bjorck(w, iters)) <= 1e-5


def test_p2_square_needs_more_iterations():
    """P2: square Gaussian matrices are orthogonal once the predicted count
    is reached (and typically not at 12-15 iterations)."""
    rng = np.random.default_rng(4)
    w = rand(rng, 64, 64)
    t_need = bjorck.iterations_to_converge(w, tol=1e-12)
    assert checks.gram_deviation(bjorck.bjorck(w, t_need + 1)) <= 1e-10
    assert checks.gram_deviation(bjorck.bjorck(w, 12)) > 1e-3


@pytest.mark.parametrize("n", [1, 4, 32])
def test_p3_orthogonal_input(n):
    """P3: an orthogonal Q has all singular values 1, so W_0 = Q / sqrt(n)
    and W_T = f^T(1/sqrt(n)) Q (scalar recursion)."""
    rng = np.random.default_rng(n)
    q, _ = np.linalg.qr(rng.standard_normal((n, n)))
    c = 1.0 / math.sqrt(n)
    for _ in range(10):
        c = 1.5 * c - 0.5 * c ** 3
    np.testing.assert_allclose(bjorck.bjorck(q, 10), c * q, rtol=0, atol=1e-13)


@pytest.mark.parametrize("rows,cols,iters", [(40, 7, 9), (7, 40, 9), (33, 1, 3), (64, 64, 12)])
def test_p3_reflected_factor_is_kept(rows, cols, iters):
    """P3 (orthogonal factor): for W = Q D with Q the first n columns of a
    Householder reflection and D diagonal, the iteration keeps Q:
    Bjorck(Q D) = Q Bjorck(D), the reference the extreme-shape GPU tests
    use (tests/reflected.py), checked against the oracle on the dense W."""
    import reflected
    v, d = reflected.factors(rows * 1000 + cols, rows, cols)
    w = reflected.matrix(v, d, rows, cols)
    q = reflected.lift(v, np.eye(len(d)))
    assert np.abs(q.T @ q - np.eye(len(d))).max() <= 1e-14      # orthonormal columns
    ref = reflected.lift(v, bjorck.bjorck(np.diag(d), iters))
    got = bjorck.bjorck(w, iters)
    np.testing.assert_allclose(got, ref if rows >= cols else ref.T, rtol=0, atol=1e-13)


def test_p4_scale_invariance():
    rng = np.random.default_rng(5)
    w = rand(rng, 24, 12)
    a = bjorck.bjorck(w, 8)
    b = bjorck.bjorck(1e3 * w, 8)
    assert checks.relative_difference(b, a) <= 1e-13


def test_degenerate_inputs():
    z, st = bjorck.bjorck(np.zeros((4, 3)), 5, return_status=True)
    assert st == bjorck.STATUS_ZERO and np.all(z == 0)
    w = np.ones((3, 3))
    w[1, 1] = np.nan
    o, st = bjorck.bjorck(w, 5, return_status=True)
    assert st == bjorck.STATUS_NONFINITE and np.all(np.isnan(o))
    # zero iterations is the pre-scaled input
    w = np.arange(6.0).reshape(2, 3) + 1
    np.testing.assert_allclose(bjorck.bjorck(w, 0), w / np.linalg.norm(w), atol=1e-16)
    with pytest.raises(ValueError):
        bjorck.bjorck(w, 3, beta=0.75)
    with pytest.raises(ValueError):
        bjorck.bjorck(w, -1)


def test_planted_mistakes_fail_p1(monkeypatch):
    """A wrong sign, a dropped term or a transposed operand in the update
    breaks the closed-form pin."""
    rng = np.random.default_rng(6)
    w = rand(rng, 12, 12)
    u, s, vt = np.linalg.svd(w)
    x = s / np.sqrt(np.sum(s * s))
    for _ in range(3):
        x = 1.5 * x - 0.5 * x ** 3
    want = (u * x) @ vt
    wrong = {
        "sign": lambda m, beta=0.5: (1 + beta) * m + beta * m @ (m.T @ m),
        "dropped": lambda m, beta=0.5: m - beta * m @ (m.T @ m),
        "transposed": lambda m, beta=0.5: (1 + beta) * m - beta * (m.T @ m) @ m,
    }
    for fn in wrong.values():
        monkeypatch.setattr(bjorck, "bjorck_step", fn)
        assert checks.relative_difference(bjorck.bjorck(w, 3), want) > 1e-3


# ------------------------------------------------------------ convolution ---

def torch_conv_circular(kernel, x, stride, dilation, groups):
    k = kernel.shape[-1]
    total = dilation * (k - 1) + 1 - stride
    pl = total // 2
    xt = F.pad(torch.from_numpy(np.asarray(x, dtype=np.float64)),
               (pl, total - pl, pl, total - pl), mode="circular")
    return F.conv2d(xt, torch.from_numpy(np.asarray(kernel, dtype=np.float64)),
                    stride=stride, dilation=dilation, groups=groups).numpy()


@pytest.mark.parametrize("cin,cout,k,s,d,g,hw", [
    (4, 6, 3, 1, 1, 1, 8), (4, 4, 3, 2, 1, 1, 8), (4, 8, 3, 1, 2, 2, 8),
    (6, 6, 5, 2, 3, 3, 12), (2, 8, 2, 2, 1, 1, 6), (3, 3, 1, 1, 1, 1, 5),
    (8, 4, 4, 2, 1, 2, 8),
])
def test_conv_matches_torch_circular(cin, cout, k, s, d, g, hw):
    rng = np.random.default_rng(7)
    kern = rng.standard_normal((cout, cin // g, k, k))
    x = rng.standard_normal((2, cin, hw, hw))
    got = conv.conv_circular(kern, x, s, d, g)
    want = torch_conv_circular(kern, x, s, d, g)
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)


@pytest.mark.parametrize("cin,cout,k,s,d,g", [(4, 6, 3, 1, 1, 1), (4, 8, 3, 2, 1, 2), (6, 6, 3, 1, 2, 3)])
def test_adjoint_inner_product(cin, cout, k, s, d, g):
    """<conv(K, x), y> == <x, conv^T(K, y)>."""
    rng = np.random.default_rng(8)
    kern = rng.standard_normal((cout, cin // g, k, k))
    x = rng.standard_normal((3, cin, 8, 8))
    y = rng.standard_normal((3, cout, 8 // s, 8 // s))
    lhs = np.sum(conv.conv_circular(kern, x, s, d, g) * y)
    rhs = np.sum(x * conv.conv_circular_adjoint(kern, y, (8, 8), s, d, g))
    assert abs(lhs - rhs) <= 1e-10 * abs(lhs)


@pytest.mark.parametrize("cin,cout,k,s,d,g,hw", [
    (4, 6, 3, 1, 1, 1, 8), (4, 4, 3, 2, 1, 1, 8), (4, 8, 3, 1, 2, 2, 8),
    (6, 6, 5, 2, 3, 3, 12), (2, 8, 2, 2, 1, 1, 6), (8, 4, 4, 2, 1, 2, 8),
])
def test_transposed_conv_matches_torch_fold(cin, cout, k, s, d, g, hw):
    """The transposed conv (adjoint) equals torch's conv_transpose2d without
    padding followed by folding its output back onto the H x W torus with
    the left padding removed: an independent route to the same operator."""
    rng = np.random.default_rng(17)
    kern = rng.standard_normal((cout, cin // g, k, k))
    y = rng.standard_normal((2, cout, hw // s, hw // s))
    full = F.conv_transpose2d(torch.from_numpy(y), torch.from_numpy(kern), stride=s, dilation=d,
                              groups=g).numpy()
    pl = (d * (k - 1) + 1 - s) // 2
    want = np.zeros((2, cin, hw, hw))
    for t in range(full.shape[2]):
        for u in range(full.shape[3]):
            want[:, :, (t - pl) % hw, (u - pl) % hw] += full[:, :, t, u]
    got = conv.conv_circular_adjoint(kern, y, (hw, hw), s, d, g)
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)


def test_transposed_toeplitz_is_transpose():
    """Impulse responses of the transposed conv give the transpose of the
    forward conv's Toeplitz matrix."""
    rng = np.random.default_rng(18)
    cin, cout, k, s, d, g, hw = 4, 6, 3, 2, 1, 2, 6
    kern = rng.standard_normal((cout, cin // g, k, k))
    fwd = conv.toeplitz_matrix(kern, hw, hw, s, d, g)
    dim = cout * (hw // s) ** 2
    basis = np.eye(dim).reshape(dim, cout, hw // s, hw // s)
    cols = conv.conv_circular_adjoint(kern, basis, (hw, hw), s, d, g).reshape(dim, -1).T
    np.testing.assert_allclose(cols, fwd.T, rtol=0, atol=1e-13)


@pytest.mark.parametrize("shape_a,shape_b,stride", [
    ((5, 4, 2, 2), (4, 3, 1, 2), 2), ((3, 4, 1, 1), (4, 4, 2, 1), 1),
    ((4, 4, 2, 3), (4, 2, 3, 2), 1),
])
def test_block_conv_is_conv_of_conv(shape_a, shape_b, stride):
    """(A ⊛ B) applied with stride s equals A (stride s) after B (stride 1),
    checked with torch's conv2d on an unpadded input."""
    rng = np.random.default_rng(9)
    a = rng.standard_normal(shape_a)
    b = rng.standard_normal(shape_b)
    x = torch.from_numpy(rng.standard_normal((2, shape_b[1], 12, 12)))
    inner = F.conv2d(x, torch.from_numpy(b))
    two = F.conv2d(inner, torch.from_numpy(a), stride=stride)
    one = F.conv2d(x, torch.from_numpy(aoc.block_conv(a, b)), stride=stride)
    np.testing.assert_allclose(one.numpy(), two.numpy(), rtol=0, atol=1e-11)


def test_p5_block_conv_algebra():
    rng = np.random.default_rng(10)
    a = rng.standard_normal((3, 4, 2, 1))
    b = rng.standard_normal((4, 5, 1, 2))
    c = rng.standard_normal((5, 2, 2, 2))
    left = aoc.block_conv(aoc.block_conv(a, b), c)
    right = aoc.block_conv(a, aoc.block_conv(b, c))
    np.testing.assert_allclose(left, right, atol=1e-12)
    np.testing.assert_allclose(aoc.block_conv(aoc.identity_kernel(3), a), a, atol=0)
    np.testing.assert_allclose(aoc.block_conv(a, aoc.identity_kernel(4)), a, atol=0)


def test_p5_projector_properties():
    rng = np.random.default_rng(12)
    v = bjorck.bjorck(rand(rng, 16, 8), 30)
    p = aoc.projector(v)
    np.testing.assert_allclose(p @ p, p, atol=1e-12)
    np.testing.assert_allclose(p, p.T, atol=0)
    assert abs(np.trace(p) - 8) <= 1e-12
    # rotation invariance (P4): V O gives the same projector
    o, _ = np.linalg.qr(rng.standard_normal((8, 8)))
    np.testing.assert_allclose(aoc.projector(v @ o), p, atol=1e-12)


def test_p5_reductions_k_equals_s():
    rng = np.random.default_rng(13)
    m = bjorck.bjorck(rand(rng, 6, 6), 40)
    k1 = aoc.aoc_kernel(m[None], None, 6, 6, 1, 1, 1, 1)
    np.testing.assert_allclose(k1[:, :, 0, 0], m, atol=0)
    m2 = bjorck.bjorck(rand(rng, 8, 12), 40)     # cout 8, c 3, s 2
    k2 = aoc.aoc_kernel(m2[None], None, 3, 8, 2, 2, 1, 1)
    np.testing.assert_allclose(k2.reshape(8, 12), m2, atol=0)


def aoc_case(rng, cin, cout, k, s, d, g, iters=60):
    rr, rc, npj, pr, pc = aoc.param_shapes(cin, cout, k, s, d, g)
    raw_r = np.stack([rand(rng, rr, rc) for _ in range(g)])
    raw_p = np.stack([np.stack([rand(rng, pr, pc) for _ in range(npj)]) for _ in range(g)]) if npj else None
    kern = aoc.aoc_layer(raw_r, raw_p, cin, cout, k, s, d, g, iters)
    mats = [bjorck.bjorck(raw_r[j], iters) for j in range(g)]
    return kern, mats


GEOMS = [(4, 4, 3, 1, 1, 1), (4, 8, 3, 2, 1, 1), (4, 4, 3, 2, 1, 1), (2, 8, 2, 2, 1, 1),
         (4, 4, 3, 1, 2, 1), (4, 16, 3, 2, 3, 1), (4, 4, 5, 1, 1, 1), (4, 6, 3, 1, 1, 1),
         (8, 8, 3, 1, 1, 2), (6, 4, 4, 2, 1, 2)]


@pytest.mark.parametrize("geom", GEOMS)
def test_p6_toeplitz_spectrum(geom):
    """P6: the spectrum of the circular convolution is the spectrum of the
    RKO matrices, each value repeated (H/s)(W/s) times (the BCOP factor is
    unitary); with converged factors every singular value is 1."""
    cin, cout, k, s, d, g = geom
    rng = np.random.default_rng(sum(geom))
    hw = 8
    kern, mats = aoc_case(rng, cin, cout, k, s, d, g)
    sv = conv.toeplitz_singular_values(kern, hw, hw, s, d, g)
    reps = (hw // s) ** 2
    want = np.sort(np.concatenate([np.repeat(np.linalg.svd(m, compute_uv=False), reps) for m in mats]))[::-1]
    np.testing.assert_allclose(sv[:want.size], want, atol=1e-8)
    np.testing.assert_allclose(sv, 1.0, atol=1e-8)


def test_p6_unconverged_spectrum_matches_matrix():
    """With converged projectors (so the BCOP factor is unitary) but an
    RKO factor stopped after 3 iterations, the conv spectrum equals that RKO
    matrix's spectrum (not 1): the construction is exact, convergence is
    the matrix iteration's business."""
    rng = np.random.default_rng(21)
    rr, rc, npj, pr, pc = aoc.param_shapes(4, 4, 3, 1, 1, 1)
    m = bjorck.bjorck(rand(rng, rr, rc), 3)
    proj = np.stack([bjorck.bjorck(rand(rng, pr, pc), 60) for _ in range(npj)])
    kern = aoc.aoc_kernel(m[None], proj[None], 4, 4, 3, 1, 1, 1)
    sv = conv.toeplitz_singular_values(kern, 8, 8)
    want = np.sort(np.repeat(np.linalg.svd(m, compute_uv=False), 64))[::-1]
    np.testing.assert_allclose(sv, want, atol=1e-10)
    assert np.max(np.abs(sv - 1)) > 1e-2


def test_stride_dilation_rejection_is_needed():
    """s = 2 with d = 2 shares input pixels between patches: the spectrum
    leaves 1, which is why such geometries are rejected (P9)."""
    rng = np.random.default_rng(22)
    rr, rc = 8, 16
    m = bjorck.bjorck(rand(rng, rr, rc), 60)
    kern = aoc.rko_kernel(m, 4, 2)        # k = s = 2: pure RKO
    sv = conv.toeplitz_singular_values(kern, 8, 8, 2, 2, 1)
    assert np.max(np.abs(sv - 1)) > 0.5


@pytest.mark.parametrize("geom", [(4, 4, 3, 1, 1, 1), (4, 4, 3, 1, 2, 1), (8, 8, 5, 1, 1, 2), (4, 6, 3, 1, 1, 1)])
def test_p7_fft_spectrum_equals_toeplitz(geom):
    cin, cout, k, s, d, g = geom
    rng = np.random.default_rng(31)
    kern, _ = aoc_case(rng, cin, cout, k, s, d, g, iters=5)
    a = conv.toeplitz_singular_values(kern, 8, 8, 1, d, g)
    b = conv.fft_singular_values(kern, 8, 8, d, g)
    np.testing.assert_allclose(a[:b.size], b, atol=1e-10)


@pytest.mark.parametrize("geom", [(16, 16, 3, 1, 1, 1), (4, 16, 3, 2, 1, 1), (8, 8, 3, 1, 2, 2),
                                  (4, 16, 2, 2, 1, 1), (4, 6, 3, 1, 1, 1)])
def test_p8_norm_preservation(geom):
    cin, cout, k, s, d, g = geom
    rng = np.random.default_rng(41)
    kern, _ = aoc_case(rng, cin, cout, k, s, d, g)
    x = rng.standard_normal((3, cin, 8, 8))
    r = checks.conv_norm_ratios(kern, x, s, d, g)
    np.testing.assert_allclose(r, 1.0, atol=1e-10)


def test_p8_wide_layer_adjoint():
    """A layer with cout/g < c s^2 is a co-isometry: its adjoint preserves norms."""
    rng = np.random.default_rng(42)
    kern, _ = aoc_case(rng, 8, 8, 3, 2, 1, 1)       # RKO 8 x 32: wide
    y = rng.standard_normal((2, 8, 4, 4))
    r = checks.conv_adjoint_norm_ratios(kern, y, (8, 8), 2, 1, 1)
    np.testing.assert_allclose(r, 1.0, atol=1e-10)


@pytest.mark.parametrize("geom,kind", [
    ((4, 4, 1, 2, 1, 1), "unsupported"),      # k < s
    ((4, 4, 3, 2, 2, 1), "unsupported"),      # gcd(s, d) != 1
    ((4, 4, 3, 1, 1, 3), "invalid"),          # groups do not divide
    ((0, 4, 3, 1, 1, 1), "invalid"),
    ((2, 4, 3, 1, 1, 2), "unsupported"),      # c = 1 with BCOP blocks
])
def test_p9_rejections(geom, kind):
    with pytest.raises(aoc.GeometryError) as e:
        aoc.validate_geometry(*geom)
    assert e.value.kind == kind


def test_param_shapes():
    assert aoc.param_shapes(16, 16, 3, 1, 1, 1) == (16, 16, 4, 16, 8)
    assert aoc.param_shapes(64, 128, 3, 2, 1, 1) == (128, 256, 2, 64, 32)
    assert aoc.param_shapes(128, 512, 2, 2, 1, 1) == (512, 512, 0, 128, 64)
    assert aoc.param_shapes(256, 256, 3, 1, 1, 4) == (64, 64, 4, 64, 32)


def test_tile_relative_differences_localizes_errors():
    """The per-tile check used by the bf16 parity tests: one wrong 32 x 32
    sub-block of a 2000 x 1100 matrix moves the whole-matrix relative
    difference by about 3% but the difference of its 256-tile by about
    18%; ragged edge tiles are covered; an exact copy gives zeros."""
    rng = np.random.default_rng(3)
    b = rng.standard_normal((2000, 1100))
    assert np.all(checks.tile_relative_differences(b.copy(), b) == 0)
    a = b.copy()
    a[512 + 64:512 + 96, 256 + 32:256 + 64] = rng.standard_normal((32, 32))
    t = checks.tile_relative_differences(a, b)
    assert t.shape == (8, 5)
    assert checks.relative_difference(a, b) < 0.04
    assert t[2, 1] > 0.15 and np.count_nonzero(t) == 1
    # the ragged bottom-right tile (208 x 76) is its own block
    a = b.copy()
    a[-1, -1] += 1.0
    t = checks.tile_relative_differences(a, b)
    assert np.count_nonzero(t) == 1 and t[7, 4] > 0
    ref = np.linalg.norm(b[1792:, 1024:])
    assert abs(t[7, 4] - 1.0 / ref) < 1e-12
