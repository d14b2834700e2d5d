"""GPU parity of the Björck vector-Jacobian product (orth_orthogonalize_vjp_batched)
against the float64 oracle (oracle/bjorck_grad.py) on the same seeded inputs.

Tolerances on the relative Frobenius difference to the oracle:
  fp32 products : 1e-5.  Replaying the recurrence in float32 arithmetic (the
                  kernel's rounding points) gives 3e-7 .. 3e-6 on the shapes
                  below; the forward's fp32 bound is kept.
  bf16 operands : the saved X_t, E_t and the gradient operands Y and S are
                  rounded to bf16 (u = 2^-9).  Replaying those roundings
                  gives 2.3e-3 .. 3.5e-3 for rectangular matrices (converged
                  at T = 20) and 1.5e-2 .. 3.2e-2 for square Gaussian ones,
                  whose smallest singular values are still far from 1 and
                  amplify the operand rounding.  Bounds: 1e-2 rectangular,
                  6e-2 square (about 2x the replayed error).
"""

import numpy as np
import pytest
import torch

from oracle import bjorck_grad, checks
from paper_2601_13776_amd import orth
from paper_2601_13776_amd import workloads as wl

from gpu_util import DEV, to_dev, to_f64

pytestmark = pytest.mark.gpu

REL_F32 = 1e-5
REL_BF16_RECT = 1e-2
REL_BF16_SQUARE = 6e-2


def stored(seed, shapes, dtype="f32"):
    w = wl.Workload("test", seed, dtype, 0, ())
    return [wl.stored_matrix(w, i, r, c) for i, (r, c) in enumerate(shapes)]


def upstream(seed, shapes):
    """dL/d(output): N(0, 1) float32 matrices."""
    rng = np.random.default_rng(seed)
    return [rng.standard_normal(s).astype(np.float32) for s in shapes]


def run_vjp(st, gouts, iters, compute="f32", beta=0.5, prescale="frobenius", gin_dtype=None):
    ws = [to_dev(s) for s in st]
    gos = [torch.from_numpy(g).to(DEV) for g in gouts]
    gis = [torch.empty(w.shape, dtype=w.dtype, device=DEV) for w in ws]
    status = torch.full((len(ws),), -1, dtype=torch.int32, device=DEV)
    orth.orth_orthogonalize_vjp_batched(ws, gos, gis, iters, beta=beta, prescale=prescale, compute=compute,
                                        status=status)
    torch.cuda.synchronize()
    return gis, status.cpu().numpy()


SHAPES_F32 = [(1, 1), (1, 7), (7, 1), (16, 8), (8, 16), (33, 17), (64, 64), (128, 64), (64, 128), (100, 50),
              (65, 65), (129, 64), (200, 130), (256, 128), (128, 256), (300, 300), (512, 256)]


@pytest.mark.parametrize("iters", [0, 1, 12])
def test_vjp_f32_mixed_batch(iters):
    print(f"[vjp f32] iters={iters}", flush=True)
    st = stored(201, SHAPES_F32)
    gouts = upstream(202, SHAPES_F32)
    gis, status = run_vjp(st, gouts, iters)
    assert np.all(status == 0)
    for s, g, o, shape in zip(st, gouts, gis, SHAPES_F32):
        ref = bjorck_grad.bjorck_vjp(wl.as_f64(s), g.astype(np.float64), iters)
        got = to_f64(o)
        assert got.shape == shape
        rel = checks.relative_difference(got, ref)
        assert rel <= REL_F32, (shape, rel)


@pytest.mark.parametrize("beta,prescale", [(0.25, "frobenius"), (0.5, "none")])
def test_vjp_f32_beta_and_no_prescale(beta, prescale):
    shapes = [(48, 20), (20, 48), (96, 96), (200, 72)]
    st = stored(203, shapes)
    if prescale == "none":   # put the inputs inside the basin without scaling
        st = [(s / np.linalg.norm(s.astype(np.float64), 2) * 0.9).astype(np.float32) for s in st]
    gouts = upstream(204, shapes)
    gis, status = run_vjp(st, gouts, 10, beta=beta, prescale=prescale)
    assert np.all(status == 0)
    for s, g, o, shape in zip(st, gouts, gis, shapes):
        ref = bjorck_grad.bjorck_vjp(s.astype(np.float64), g.astype(np.float64), 10, beta, prescale)
        assert checks.relative_difference(to_f64(o), ref) <= REL_F32, shape


SHAPES_BF16 = [(128, 64), (64, 100), (256, 128), (300, 700), (1024, 512), (256, 256), (512, 512), (1100, 1030)]


def test_vjp_bf16_mixed_batch():
    """bf16 parameters, fp32 upstream gradient, bf16 products (the small
    bucket runs in fp32 as in the forward)."""
    print("[vjp bf16] mixed batch", flush=True)
    st = stored(205, SHAPES_BF16, "bf16")
    gouts = upstream(206, SHAPES_BF16)
    gis, status = run_vjp(st, gouts, 20, compute="bf16")
    assert np.all(status == 0)
    for s, g, o, shape in zip(st, gouts, gis, SHAPES_BF16):
        assert o.dtype == torch.bfloat16
        ref = bjorck_grad.bjorck_vjp(wl.as_f64(s), g.astype(np.float64), 20)
        rel = checks.relative_difference(to_f64(o), ref)
        bound = REL_BF16_SQUARE if shape[0] == shape[1] else REL_BF16_RECT
        assert rel <= bound, (shape, rel)


def test_vjp_scale_invariance_property():
    """With Frobenius pre-scaling the gradient is orthogonal to W (any size)."""
    shapes = [(384, 200), (200, 384), (2048, 1024)]
    st = stored(207, shapes, "bf16")
    gouts = upstream(208, shapes)
    gis, _ = run_vjp(st, gouts, 15, compute="bf16")
    for s, o in zip(st, gis):
        w, g = wl.as_f64(s), to_f64(o)
        assert abs(float(np.sum(w * g))) <= 1e-2 * np.linalg.norm(w) * np.linalg.norm(g)


def test_vjp_statuses_and_empty():
    shapes = [(40, 20), (40, 20), (20, 40), (300, 200)]
    st = stored(209, shapes)
    st[1] = np.zeros_like(st[1])
    st[2] = st[2].copy()
    st[2][3, 5] = np.nan
    gouts = upstream(210, shapes)
    gis, status = run_vjp(st, gouts, 6)
    assert list(status) == [0, 1, 2, 0]
    assert torch.all(gis[1] == 0)
    assert torch.all(torch.isnan(gis[2]))
    for i in (0, 3):
        ref = bjorck_grad.bjorck_vjp(st[i].astype(np.float64), gouts[i].astype(np.float64), 6)
        assert checks.relative_difference(to_f64(gis[i]), ref) <= REL_F32
    # an empty batch launches nothing
    assert orth.orth_orthogonalize_vjp_batched([], [], [], 6) is None


@pytest.mark.parametrize("alias", ["grad_out", "w"])
def test_vjp_aliasing_and_strides(alias):
    shapes = [(90, 40), (40, 90), (260, 130)]
    st = stored(211, shapes)
    gouts = upstream(212, shapes)
    refs = [bjorck_grad.bjorck_vjp(s.astype(np.float64), g.astype(np.float64), 8) for s, g in zip(st, gouts)]
    ws, gos, gis = [], [], []
    for s, g in zip(st, gouts):
        # strided views: leading dimension larger than cols
        big = torch.zeros(s.shape[0], s.shape[1] + 24, device=DEV)
        big[:, :s.shape[1]] = torch.from_numpy(s)
        w = big[:, :s.shape[1]]
        bg = torch.zeros(s.shape[0], s.shape[1] + 24, device=DEV)
        bg[:, :s.shape[1]] = torch.from_numpy(g)
        go = bg[:, :s.shape[1]]
        ws.append(w)
        gos.append(go)
        gis.append(go if alias == "grad_out" else w)
    orth.orth_orthogonalize_vjp_batched(ws, gos, gis, 8)
    torch.cuda.synchronize()
    for o, ref, shape in zip(gis, refs, shapes):
        assert checks.relative_difference(to_f64(o), ref) <= REL_F32, shape
