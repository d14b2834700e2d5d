"""Pins of the spectral pre-scaling oracle (oracle/spectral.py):

S1  hand-derived cases on small diagonal matrices (tests/golden/spectral_hand.json);
S2  with enough power steps the estimate reaches the SVD's largest singular
    value and the vector its right singular vector (numpy SVD);
S3  bounds that hold for any cached vector: ||X v|| <= sigma_hat and
    sigma <= sigma_max (so the largest singular value of W_0 is >= 1);
S4  the wide case is the transpose of the tall case;
S5  the point of the step: from a good cached vector, spectral scaling
    needs fewer Björck iterations than Frobenius scaling, about
    log_1.5(||W||_F / sigma) fewer on the workload's matrices;
S6  statuses, and planted mistakes that the pins catch;
S7  the vector-Jacobian product through the pre-scaling (cached vector held
    constant): central finite differences of the oracle forward in both
    branches of the max, every Jacobian entry on tiny matrices; torch
    autograd through an independent float64 torch forward of the power
    steps and the iteration; the statuses; planted mistakes (the earlier
    power steps' dependence on W dropped, the other branch's derivative)
    that the finite differences catch.
"""

import json
import math
import os
import zlib

import numpy as np
import pytest

from oracle import bjorck, spectral

HERE = os.path.dirname(os.path.abspath(__file__))
RNG = np.random.default_rng(20260114)


@pytest.fixture(autouse=True)
def _rng_per_test(request):
    """Each test draws from a generator seeded by its own name, so that its
    inputs do not depend on which tests ran before it in the process (a
    parallel run deals tests to workers in any order)."""
    global RNG
    RNG = np.random.default_rng([20260114, zlib.crc32(request.node.name.encode())])


def ev(expr):
    return float(eval(expr, {"sqrt": math.sqrt}))


CASES = json.load(open(os.path.join(HERE, "golden", "spectral_hand.json")))["cases"]


@pytest.mark.parametrize("case", CASES, ids=[c["name"] for c in CASES])
def test_hand_cases(case):
    w = np.array(case["w"], dtype=np.float64)
    w0, v, sigma, status = spectral.spectral_prescale(w, case["u"], case["q"])
    assert status == bjorck.STATUS_OK
    assert abs(sigma - ev(case["sigma"])) <= 1e-14 * ev(case["sigma"])
    np.testing.assert_allclose(v, [ev(e) for e in case["v"]], rtol=0, atol=1e-15)
    np.testing.assert_allclose(w0, w / ev(case["sigma"]), rtol=1e-14, atol=0)


@pytest.mark.parametrize("shape", [(40, 12), (12, 40), (30, 30)])
def test_converges_to_svd(shape):
    w = RNG.standard_normal(shape)
    u, s, vt = np.linalg.svd(w if shape[0] >= shape[1] else w.T)
    # enough steps for (s1 / s0)^(2 q) <= 1e-14, the power method's rate
    q = int(np.ceil(14 * np.log(10) / (2 * np.log(s[0] / s[1])))) + 10
    _, v, sigma, _ = spectral.spectral_prescale(w, RNG.standard_normal(min(shape)), q)
    assert abs(sigma - s[0]) <= 1e-9 * s[0]
    assert abs(abs(float(v @ vt[0])) - 1.0) <= 1e-9


@pytest.mark.parametrize("q", [1, 2, 5])
def test_bounds_any_vector(q):
    for _ in range(20):
        m, n = RNG.integers(2, 30, size=2)
        w = RNG.standard_normal((m, n)) * RNG.uniform(0.01, 100)
        x_mat = w if m >= n else w.T
        u = RNG.standard_normal(min(m, n))
        w0, v, sigma, _ = spectral.spectral_prescale(w, u, q)
        smax = np.linalg.svd(w, compute_uv=False)[0]
        # both sigma_hat and ||W||_F / sqrt(N) are lower bounds of sigma_max
        assert sigma <= smax * (1 + 1e-12)
        assert sigma >= np.linalg.norm(w) / math.sqrt(min(m, n)) * (1 - 1e-12)
        assert np.linalg.svd(w0, compute_uv=False)[0] >= 1 - 1e-12
        # one step from a unit vector: sigma_hat >= ||X v_in||
        uin = u / np.linalg.norm(u)
        _, _, s1, _ = spectral.spectral_prescale(w, u, 1)
        assert s1 >= np.linalg.norm(x_mat @ uin) * (1 - 1e-12)
        assert abs(np.linalg.norm(v) - 1.0) <= 1e-12


def test_transpose_relation():
    w = RNG.standard_normal((9, 21))
    u = RNG.standard_normal(9)
    a0, av, asig, _ = spectral.spectral_prescale(w, u, 3)
    b0, bv, bsig, _ = spectral.spectral_prescale(w.T, u, 3)
    assert asig == pytest.approx(bsig, rel=1e-14)
    np.testing.assert_allclose(a0, b0.T, rtol=1e-14)
    np.testing.assert_allclose(av, bv, rtol=1e-13, atol=1e-15)


@pytest.mark.parametrize("n", [64, 128])
def test_fewer_iterations_than_frobenius(n):
    """Square Gaussian matrices: with the cached top vector (a previous
    step's result), one power step gives sigma close to sigma_max and the
    iteration converges in fewer steps than after Frobenius scaling."""
    w = RNG.standard_normal((n, n)) / math.sqrt(n)
    _, cached, _, _ = spectral.spectral_prescale(w, RNG.standard_normal(n), 30)
    w_next = w + 1e-3 * RNG.standard_normal((n, n)) / math.sqrt(n)   # a small parameter update
    _, _, sigma, _ = spectral.spectral_prescale(w_next, cached, 1)
    t_spec = spectral.iterations_to_converge_scaled(w_next, sigma, tol=1e-3)
    t_frob = spectral.iterations_to_converge_scaled(w_next, np.linalg.norm(w_next), tol=1e-3)
    assert t_spec is not None and t_frob is not None
    assert t_spec + 3 <= t_frob


def test_bjorck_spectral_and_statuses():
    w = RNG.standard_normal((20, 8))
    out, v, st = spectral.bjorck_spectral(w, np.ones(8), 30, 2)
    assert st == 0
    assert np.max(np.abs(out.T @ out - np.eye(8))) <= 1e-10
    z, vz, st = spectral.bjorck_spectral(np.zeros((5, 3)), np.arange(3.0), 4)
    assert st == bjorck.STATUS_ZERO and np.all(z == 0) and np.array_equal(vz, np.arange(3.0))
    bad = w.copy()
    bad[0, 0] = np.nan
    o, vb, st = spectral.bjorck_spectral(bad, np.ones(8), 4)
    assert st == bjorck.STATUS_NONFINITE and np.all(np.isnan(o)) and np.array_equal(vb, np.ones(8))
    with pytest.raises(ValueError):
        spectral.spectral_prescale(w, np.ones(8), 0)


def test_planted_missing_lower_bound(monkeypatch):
    """Without max(., ||W||_F / sqrt(N)) a cached vector in the null space of
    the top direction leaves W_0 outside the basin (0, sqrt(3)); with it the
    hand case "null-space start" stays inside."""
    w = np.diag([10.0, 1.0, 1.0])
    u = np.array([0.0, 1.0, 1.0])
    w0, _, _, _ = spectral.spectral_prescale(w, u, 1)
    assert np.linalg.svd(w0, compute_uv=False)[0] < math.sqrt(3)
    orig = spectral.spectral_prescale

    def no_bound(w, u, q):
        w0, v, sigma, st = orig(w, u, q)
        x_mat = w if w.shape[0] >= w.shape[1] else w.T
        x = x_mat @ (u / np.linalg.norm(u))
        y = x_mat.T @ x
        s_hat = np.linalg.norm(y) / np.linalg.norm(x)
        return w / s_hat, v, s_hat, st
    monkeypatch.setattr(spectral, "spectral_prescale", no_bound)
    w0, _, _, _ = spectral.spectral_prescale(w, u, 1)
    assert np.linalg.svd(w0, compute_uv=False)[0] > math.sqrt(3)
    with pytest.raises(AssertionError):
        test_hand_cases(CASES[4])


def test_planted_norm_instead_of_ratio(monkeypatch):
    """Using ||X v|| instead of ||X^T X v|| / ||X v|| fails the hand case."""
    def wrong(w, u, q):
        x_mat = w if w.shape[0] >= w.shape[1] else w.T
        v = np.asarray(u, float) / np.linalg.norm(u)
        s = np.linalg.norm(x_mat @ v)
        sigma = max(s, np.linalg.norm(w) / math.sqrt(min(w.shape)))
        return w / sigma, v, sigma, 0
    monkeypatch.setattr(spectral, "spectral_prescale", wrong)
    with pytest.raises(AssertionError):
        test_hand_cases(CASES[2])


def test_workload_shapes_step_saving():
    """On matrices of the ImageNet-like stack (seeded as the workload draws
    them): in the linear phase of the scalar map (small singular values grow
    by 1.5 per step) spectral scaling starts every singular value
    ||W||_F / sigma times larger than Frobenius scaling does, which saves
    about log_1.5(||W||_F / sigma) steps.  Spectral scaling from a warmed
    vector at T - (that count, rounded down, minus one) is at least as
    orthogonal as Frobenius scaling at T = 20."""
    from paper_2601_13776_amd import workloads as wl
    w = wl.WORKLOADS["imagenet_backbone25"]
    shapes = w.matrix_shapes()
    saved = []
    for i in (0, 1, 20, 61, 80):   # 128^2, 128x64, 256^2, 1024x512, dense 1024^2
        x = wl.as_f64(wl.stored_matrix(w, i, *shapes[i]))
        _, warm, _, _ = spectral.spectral_prescale(x, np.ones(min(x.shape)), 20)
        _, _, sigma, _ = spectral.spectral_prescale(x, warm, 1)
        k = int(math.floor(math.log(np.linalg.norm(x) / sigma, 1.5))) - 1
        spec, _, _ = spectral.bjorck_spectral(x, warm, 20 - k, 1)
        frob = bjorck.bjorck(x, 20)
        dev = lambda m: np.max(np.abs((m.T @ m if m.shape[0] >= m.shape[1] else m @ m.T) - np.eye(min(m.shape))))
        assert dev(spec) <= max(dev(frob), 1e-12), (i, shapes[i], k, dev(spec), dev(frob))
        saved.append(k)
    assert min(saved) >= 2 and max(saved) >= 5


# ------------------------------------------------------------------ S7 ---
def fd_spectral(w, u, y, d, iters, q, h=1e-6):
    """The directional derivative of <Y, Bjorck(W / sigma)> along D (the
    cached vector u held constant) by central differences at steps h and
    h/2, combined so that their second-order truncation terms cancel, and a
    bound on its error: the two differences' gap plus the rounding of the
    function values (a few machine epsilons of their absolute sums, over
    the step).  Returns (estimate, error bound)."""
    f = lambda x: spectral.bjorck_spectral(x, u, iters, q)[0]
    v = {t: y * f(w + t * d) for t in (h, -h, h / 2, -h / 2)}
    d1 = float(np.sum(v[h] - v[-h])) / (2 * h)
    d2 = float(np.sum(v[h / 2] - v[-h / 2])) / h
    rounding = 8 * np.finfo(np.float64).eps * max(float(np.sum(np.abs(a))) for a in v.values()) / h
    return (4 * d2 - d1) / 3, abs(d2 - d1) + rounding


def assert_fd(gd, fd_err, rel):
    """<G, D> agrees with the finite difference to `rel` (relative) beyond
    the difference's own error bound, which must itself be small enough for
    the check to mean something."""
    fd, err = fd_err
    assert err <= 1e-5 * max(1.0, abs(fd)), (fd, err)
    assert abs(gd - fd) <= rel * max(1.0, abs(fd)) + err, (gd, fd, err)


def frobenius_branch_case(rng, n=5):
    """A matrix whose power-iteration estimate from the cached vector stays
    below ||W||_F / sqrt(N): the cached vector lies on a small singular
    direction of a matrix with one large singular value (the perturbation is
    small enough that q <= 2 power steps stay below the bound whatever it
    draws: the top direction's share grows about 16-fold per step)."""
    w = np.diag([4.0] + [1.0] * (n - 1)) + 0.001 * rng.standard_normal((n, n))
    u = np.zeros(n)
    u[1] = 1.0
    return w, u


@pytest.mark.parametrize("shape,q", [((7, 4), 1), ((7, 4), 3), ((4, 7), 2), ((6, 6), 1), ((6, 6), 4), ((9, 1), 2)])
def test_spectral_vjp_directional_fd(shape, q):
    w = RNG.standard_normal(shape)
    # a warmed cached vector (as in training): the power-iteration branch
    u = spectral.spectral_prescale(w, RNG.standard_normal(min(shape)), 30)[1]
    y = RNG.standard_normal(shape)
    _, _, sigma, _ = spectral.spectral_prescale(w, u, q)
    # power-iteration branch (with one column the two bounds are the same
    # function, ||W||, and tie up to rounding)
    assert sigma > np.linalg.norm(w) / np.sqrt(min(shape)) * (1 - (1e-12 if min(shape) == 1 else 0))
    g = spectral.bjorck_spectral_vjp(w, u, y, 5, q)
    for _ in range(3):
        d = RNG.standard_normal(shape)
        assert_fd(float(np.sum(g * d)), fd_spectral(w, u, y, d, 5, q), 1e-7)


@pytest.mark.parametrize("q", [1, 2])
def test_spectral_vjp_frobenius_branch_fd(q):
    w, u = frobenius_branch_case(RNG)
    _, _, sigma, _ = spectral.spectral_prescale(w, u, q)
    assert sigma == np.linalg.norm(w) / np.sqrt(5)
    y = RNG.standard_normal(w.shape)
    g = spectral.bjorck_spectral_vjp(w, u, y, 4, q)
    for _ in range(3):
        d = RNG.standard_normal(w.shape)
        assert_fd(float(np.sum(g * d)), fd_spectral(w, u, y, d, 4, q), 1e-7)


def test_spectral_vjp_full_jacobian_fd():
    w = RNG.standard_normal((3, 2))
    u = RNG.standard_normal(2)
    y = RNG.standard_normal((3, 2))
    g = spectral.bjorck_spectral_vjp(w, u, y, 3, 2)
    for i in range(3):
        for j in range(2):
            e = np.zeros(w.shape)
            e[i, j] = 1.0
            assert_fd(g[i, j], fd_spectral(w, u, y, e, 3, 2), 1e-8)


def torch_spectral_forward(w, u, iters, q, beta=0.5):
    """Power steps and iteration written with torch ops (test-local)."""
    import torch
    tall = w.shape[0] >= w.shape[1]
    x_mat = w if tall else w.mT
    v = u / torch.linalg.vector_norm(u)
    for _ in range(q):
        x = x_mat @ v
        y = x_mat.mT @ x
        sig = torch.linalg.vector_norm(y) / torch.linalg.vector_norm(x)
        v = y / torch.linalg.vector_norm(y)
    floor = torch.linalg.matrix_norm(w) / min(w.shape) ** 0.5
    z = w / (sig if sig >= floor else floor)
    for _ in range(iters):
        z = (1 + beta) * z - beta * (z @ z.mT @ z)
    return z


@pytest.mark.parametrize("shape,q,branch", [((12, 5), 2, "power"), ((5, 12), 3, "power"), ((8, 8), 1, "power"),
                                            ((5, 5), 2, "frobenius")])
def test_spectral_vjp_matches_torch_autograd(shape, q, branch):
    import torch
    if branch == "power":
        w = RNG.standard_normal(shape)
        u = RNG.standard_normal(min(shape))
    else:
        w, u = frobenius_branch_case(RNG)
    y = RNG.standard_normal(w.shape)
    wt = torch.tensor(w, dtype=torch.float64, requires_grad=True)
    out = torch_spectral_forward(wt, torch.tensor(u, dtype=torch.float64), 6, q)
    (out * torch.tensor(y)).sum().backward()
    g = spectral.bjorck_spectral_vjp(w, u, y, 6, q)
    assert np.max(np.abs(g - wt.grad.numpy())) <= 1e-10 * max(1.0, np.max(np.abs(g)))


def test_spectral_vjp_statuses():
    u = np.ones(3)
    y = RNG.standard_normal((4, 3))
    assert np.all(spectral.bjorck_spectral_vjp(np.zeros((4, 3)), u, y, 3, 1) == 0)
    bad = RNG.standard_normal((4, 3))
    bad[1, 2] = np.inf
    assert np.all(np.isnan(spectral.bjorck_spectral_vjp(bad, u, y, 3, 1)))
    # a zero cached vector starts from ones, as in the forward
    w = RNG.standard_normal((4, 3))
    g0 = spectral.bjorck_spectral_vjp(w, np.zeros(3), y, 3, 2)
    g1 = spectral.bjorck_spectral_vjp(w, np.ones(3), y, 3, 2)
    assert np.array_equal(g0, g1)


def test_planted_spectral_vjp_mistakes():
    """Treating the earlier power steps' vectors as constants, or taking the
    Frobenius branch's derivative where sigma_hat is the maximum, both
    fail the finite differences."""
    w = RNG.standard_normal((6, 4))
    u = RNG.standard_normal(4)
    y = RNG.standard_normal((6, 4))
    d = RNG.standard_normal((6, 4))
    fd, err = fd_spectral(w, u, y, d, 4, 3)
    good = float(np.sum(spectral.bjorck_spectral_vjp(w, u, y, 4, 3) * d))
    assert_fd(good, (fd, err), 1e-7)
    # only the last power step differentiated: q = 3 seen as one step from v_2
    w0, v, sigma, _ = spectral.spectral_prescale(w, u, 2)
    from oracle import bjorck_grad
    g0 = bjorck_grad.bjorck_vjp(spectral.spectral_prescale(w, u, 3)[0], y, 4, prescale="none")
    last_only = spectral.spectral_prescale_vjp(w, v, 1, g0)
    assert abs(float(np.sum(last_only * d)) - fd) > 1e-4 * max(1.0, abs(fd))
    # Frobenius branch's derivative in the power-iteration branch
    n = 4
    c = -float(np.sum(g0 * w)) / spectral.spectral_prescale(w, u, 3)[2] ** 2
    wrong = g0 / spectral.spectral_prescale(w, u, 3)[2] + c * w / (np.linalg.norm(w) * np.sqrt(n))
    assert abs(float(np.sum(wrong * d)) - fd) > 1e-4 * max(1.0, abs(fd))
