"""Pins of the oracle's vector-Jacobian products (oracle/bjorck_grad.py,
oracle/aoc_grad.py) against what does not depend on the hand derivation:

G1  central finite differences of the oracle forward, every entry of the
    Jacobian on tiny matrices and random directions on larger ones;
G2  torch.autograd through an independent float64 torch forward of the
    Appendix A.5 iteration;
G3  scale invariance: with Frobenius pre-scaling the output does not change
    along W, so the gradient is orthogonal to W;
G4  transposition: the wide case is the transpose of the tall case;
G5  the adjoint identity of the composition's part that is linear in the
    RKO factor; finite differences in the projector factors and through a
    whole layer (Björck included);
G6  planted mistakes (a dropped term, a missing symmetrization, a flipped
    sign) that each fail one of the pins above.
"""

import zlib

import numpy as np
import pytest
import torch

from oracle import aoc, aoc_grad, bjorck, bjorck_grad

RNG = np.random.default_rng(20260113)


@pytest.fixture(autouse=True)
def _rng_per_test(request):
    """Each test draws from a generator seeded by its own name, so that its
    inputs do not depend on which tests ran before it in the process (a
    parallel run deals tests to workers in any order)."""
    global RNG
    RNG = np.random.default_rng([20260113, zlib.crc32(request.node.name.encode())])


EPS = np.finfo(np.float64).eps


def fd_directional(f, w, y, d, h=1e-5):
    """The directional derivative of L = <Y, f(W)> along D by central
    differences at steps h and h/2, combined so that their second-order
    truncation terms cancel, and a bound on its error: the two central
    differences' gap (three quarters of the step-h truncation term, far
    above the combination's) plus the rounding of the function values (a
    few machine epsilons of their absolute sums, over the step).  Returns
    (estimate, error bound)."""
    v = {t: y * f(w + t * d) for t in (h, -h, h / 2, -h / 2)}
    d1 = float(np.sum(v[h] - v[-h])) / (2 * h)
    d2 = float(np.sum(v[h / 2] - v[-h / 2])) / h
    rounding = 8 * EPS * max(float(np.sum(np.abs(a))) for a in v.values()) / h
    return (4 * d2 - d1) / 3, abs(d2 - d1) + rounding


def assert_fd(gd, fd_err, rel):
    """<G, D> agrees with the finite difference to `rel` (relative) beyond
    the difference's own error bound, which must itself be small enough for
    the check to mean something."""
    fd, err = fd_err
    assert err <= 1e-5 * max(1.0, abs(fd)), (fd, err)
    assert abs(gd - fd) <= rel * max(1.0, abs(fd)) + err, (gd, fd, err)


# ----------------------------------------------------------------- G1 ---
@pytest.mark.parametrize("shape,iters", [((3, 2), 3), ((2, 3), 3), ((3, 3), 4), ((4, 1), 2)])
def test_bjorck_vjp_full_jacobian_fd(shape, iters):
    w = RNG.standard_normal(shape)
    y = RNG.standard_normal(shape)
    g = bjorck_grad.bjorck_vjp(w, y, iters)
    f = lambda x: bjorck.bjorck(x, iters)
    for i in range(shape[0]):
        for j in range(shape[1]):
            e = np.zeros(shape)
            e[i, j] = 1.0
            assert_fd(g[i, j], fd_directional(f, w, y, e), 1e-8)


@pytest.mark.parametrize("shape,iters,beta,prescale", [
    ((24, 10), 12, 0.5, "frobenius"),
    ((10, 24), 12, 0.5, "frobenius"),
    ((16, 16), 15, 0.5, "frobenius"),
    ((20, 7), 6, 0.25, "frobenius"),
    ((12, 9), 5, 0.5, "none"),
])
def test_bjorck_vjp_directional_fd(shape, iters, beta, prescale):
    w = RNG.standard_normal(shape)
    if prescale == "none":
        w = w / np.linalg.norm(w, 2) * 0.9     # inside the basin without scaling
    y = RNG.standard_normal(shape)
    g = bjorck_grad.bjorck_vjp(w, y, iters, beta, prescale)
    f = lambda x: bjorck.bjorck(x, iters, beta, prescale)
    for _ in range(4):
        d = RNG.standard_normal(shape)
        assert_fd(float(np.sum(g * d)), fd_directional(f, w, y, d), 1e-7)


# ----------------------------------------------------------------- G2 ---
def torch_bjorck(w, iters, beta, prescale):
    """The Appendix A.5 iteration written with torch ops (test-local)."""
    x = w / torch.linalg.matrix_norm(w) if prescale == "frobenius" else w
    for _ in range(iters):
        x = (1 + beta) * x - beta * (x @ x.mT @ x)
    return x


@pytest.mark.parametrize("shape,iters,beta,prescale", [
    ((33, 17), 0, 0.5, "frobenius"),
    ((33, 17), 1, 0.5, "frobenius"),
    ((17, 33), 7, 0.5, "frobenius"),
    ((40, 40), 20, 0.5, "frobenius"),
    ((64, 32), 25, 0.3, "frobenius"),
    ((30, 12), 9, 0.5, "none"),
])
def test_bjorck_vjp_vs_torch_autograd(shape, iters, beta, prescale):
    w = RNG.standard_normal(shape)
    if prescale == "none":
        w = w / np.linalg.norm(w, 2) * 0.9
    y = RNG.standard_normal(shape)
    wt = torch.tensor(w, dtype=torch.float64, requires_grad=True)
    out = torch_bjorck(wt, iters, beta, prescale)
    out.backward(torch.tensor(y, dtype=torch.float64))
    ref = wt.grad.numpy()
    got = bjorck_grad.bjorck_vjp(w, y, iters, beta, prescale)
    assert np.max(np.abs(got - ref)) <= 1e-10 * max(1.0, np.max(np.abs(ref)))


# ----------------------------------------------------------------- G3/G4 ---
@pytest.mark.parametrize("shape,iters", [((20, 8), 3), ((8, 20), 10), ((12, 12), 10)])
def test_bjorck_vjp_scale_invariance(shape, iters):
    """Unconverged (3 steps) as well as converged iterates: only the
    pre-scaling makes the output scale invariant at 3 steps."""
    w = RNG.standard_normal(shape)
    y = RNG.standard_normal(shape)
    g = bjorck_grad.bjorck_vjp(w, y, iters)
    assert abs(float(np.sum(g * w))) <= 1e-12 * np.linalg.norm(g) * np.linalg.norm(w)
    # scaling W by c scales the gradient by 1/c
    g2 = bjorck_grad.bjorck_vjp(3.0 * w, y, iters)
    assert np.max(np.abs(3.0 * g2 - g)) <= 1e-12 * np.max(np.abs(g))


def test_bjorck_vjp_transpose():
    w = RNG.standard_normal((15, 6))
    y = RNG.standard_normal((15, 6))
    g = bjorck_grad.bjorck_vjp(w, y, 8)
    gt = bjorck_grad.bjorck_vjp(w.T, y.T, 8)
    assert np.max(np.abs(g - gt.T)) <= 1e-12 * np.max(np.abs(g))


def test_bjorck_vjp_statuses():
    y = RNG.standard_normal((5, 3))
    assert np.all(bjorck_grad.bjorck_vjp(np.zeros((5, 3)), y, 4) == 0.0)
    w = RNG.standard_normal((5, 3))
    w[2, 1] = np.inf
    assert np.all(np.isnan(bjorck_grad.bjorck_vjp(w, y, 4)))
    assert np.all(np.isnan(bjorck_grad.bjorck_vjp(w, y, 4, prescale="none")))


def test_bjorck_vjp_linear_in_upstream():
    w = RNG.standard_normal((9, 5))
    y1, y2 = RNG.standard_normal((2, 9, 5))
    g = bjorck_grad.bjorck_vjp(w, 2.0 * y1 - y2, 6)
    ref = 2.0 * bjorck_grad.bjorck_vjp(w, y1, 6) - bjorck_grad.bjorck_vjp(w, y2, 6)
    assert np.max(np.abs(g - ref)) <= 1e-12 * np.max(np.abs(ref))


# ----------------------------------------------------------------- G5 ---
GEOMS = [  # (cin, cout, k, stride, dilation, groups)
    (4, 4, 3, 1, 1, 1),
    (4, 8, 3, 2, 1, 1),
    (6, 6, 3, 1, 1, 2),
    (4, 4, 2, 2, 1, 1),
    (6, 3, 4, 2, 1, 1),
    (5, 5, 3, 1, 2, 1),
]


def random_factors(cin, cout, k, s, d, g, iters=30):
    rr, rc, nproj, pr, pc = aoc.param_shapes(cin, cout, k, s, d, g)
    raw_rko = RNG.standard_normal((g, rr, rc))
    raw_proj = RNG.standard_normal((g, nproj, pr, pc)) if nproj else None
    rko = np.stack([bjorck.bjorck(raw_rko[j], iters) for j in range(g)])
    proj = None
    if nproj:
        proj = np.stack([np.stack([bjorck.bjorck(raw_proj[j, t], iters) for t in range(nproj)])
                         for j in range(g)])
    return raw_rko, raw_proj, rko, proj


@pytest.mark.parametrize("geom", GEOMS)
def test_compose_vjp_adjoint_identity_in_rko(geom):
    cin, cout, k, s, d, g = geom
    _, _, rko, proj = random_factors(*geom)
    c = cin // g
    dk = RNG.standard_normal((cout, c, k, k))
    drko, _ = aoc_grad.aoc_kernel_vjp(rko, proj, *geom, dk)
    r2 = RNG.standard_normal(rko.shape)           # any RKO values: K is linear in them
    lhs = float(np.sum(dk * aoc.aoc_kernel(r2, proj, *geom)))
    rhs = float(np.sum(drko * r2))
    assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(lhs))


@pytest.mark.parametrize("geom", [gm for gm in GEOMS if gm[2] > gm[3]])
def test_compose_vjp_fd_in_projectors(geom):
    cin, cout, k, s, d, g = geom
    _, _, rko, proj = random_factors(*geom)
    c = cin // g
    dk = RNG.standard_normal((cout, c, k, k))
    _, dproj = aoc_grad.aoc_kernel_vjp(rko, proj, *geom, dk)
    f = lambda p: aoc.aoc_kernel(rko, p, *geom)
    for _ in range(3):
        dirn = RNG.standard_normal(proj.shape)
        assert_fd(float(np.sum(dproj * dirn)), fd_directional(f, proj, dk, dirn), 1e-8)


@pytest.mark.parametrize("geom", GEOMS)
def test_layer_vjp_fd_and_scale_invariance(geom):
    cin, cout, k, s, d, g = geom
    iters = 12
    raw_rko, raw_proj, _, _ = random_factors(*geom)
    c = cin // g
    dk = RNG.standard_normal((cout, c, k, k))
    g_rko, g_proj = aoc_grad.aoc_layer_vjp(raw_rko, raw_proj, *geom, iters, dk)
    f_r = lambda r: aoc.aoc_layer(r, raw_proj, *geom, iters)
    dirn = RNG.standard_normal(raw_rko.shape)
    assert_fd(float(np.sum(g_rko * dirn)), fd_directional(f_r, raw_rko, dk, dirn), 1e-7)
    for j in range(g):
        assert abs(float(np.sum(g_rko[j] * raw_rko[j]))) <= 1e-11 * max(1.0, np.linalg.norm(g_rko[j]))
    if g_proj is not None:
        f_p = lambda p: aoc.aoc_layer(raw_rko, p, *geom, iters)
        dirn = RNG.standard_normal(raw_proj.shape)
        assert_fd(float(np.sum(g_proj * dirn)), fd_directional(f_p, raw_proj, dk, dirn), 1e-7)
        for j in range(g):
            for t in range(raw_proj.shape[1]):
                assert abs(float(np.sum(g_proj[j, t] * raw_proj[j, t]))) <= \
                    1e-11 * max(1.0, np.linalg.norm(g_proj[j, t]))


def test_compose_vjp_identity_composition():
    """k = s = 1 with an identity-shaped RKO: K is the RKO matrix itself, so
    the gradient is dK reshaped."""
    rko = RNG.standard_normal((1, 5, 5))
    dk = RNG.standard_normal((5, 5, 1, 1))
    drko, dproj = aoc_grad.aoc_kernel_vjp(rko, None, 5, 5, 1, 1, 1, 1, dk)
    assert dproj is None
    assert np.array_equal(drko[0], dk[:, :, 0, 0])


# ----------------------------------------------------------------- G6 ---
def test_planted_dropped_symmetric_term(monkeypatch):
    def wrong_step(w, y, beta=0.5):     # drops Y^T W from the symmetric factor
        g = w.T @ w
        return (1 + beta) * y - beta * (y @ g) - beta * (w @ (w.T @ y))
    monkeypatch.setattr(bjorck_grad, "bjorck_step_vjp", wrong_step)
    with pytest.raises(AssertionError):
        test_bjorck_vjp_directional_fd((24, 10), 12, 0.5, "frobenius")


def test_planted_dropped_prescale_projection(monkeypatch):
    orig = bjorck_grad.bjorck_vjp

    def wrong(w, y, iters, beta=0.5, prescale="frobenius"):
        s = np.linalg.norm(w)        # the chain through 1/||W|| forgotten
        return orig(w / s, y, iters, beta, "none") / s
    monkeypatch.setattr(bjorck_grad, "bjorck_vjp", wrong)
    with pytest.raises(AssertionError):
        test_bjorck_vjp_scale_invariance((20, 8), 3)


def test_planted_unsymmetrized_projector(monkeypatch):
    monkeypatch.setattr(aoc_grad, "projector_vjp", lambda v, dp: 2.0 * dp @ v)
    with pytest.raises(AssertionError):
        test_compose_vjp_fd_in_projectors((4, 4, 3, 1, 1, 1))


def test_planted_block_sign(monkeypatch):
    monkeypatch.setattr(aoc_grad, "block_v_vjp", lambda db: db[:, :, 0, 0] + db[:, :, 1, 0])
    with pytest.raises(AssertionError):
        test_compose_vjp_fd_in_projectors((4, 4, 3, 1, 1, 1))


def test_planted_block_conv_tap_flip(monkeypatch):
    def wrong(a, b, dc):
        da, db = orig(a, b, dc)
        return np.flip(da, axis=(2, 3)), db
    orig = aoc_grad.block_conv_vjp
    monkeypatch.setattr(aoc_grad, "block_conv_vjp", wrong)
    with pytest.raises(AssertionError):
        test_compose_vjp_adjoint_identity_in_rko((4, 8, 3, 2, 1, 1))
