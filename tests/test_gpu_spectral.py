"""GPU parity of spectral pre-scaling (prescale="spectral": power iteration
from caller-owned cached vectors, then Björck) against the float64 oracle
(oracle/spectral.py).  Outputs: the Björck tolerances (fp32 products 1e-5,
bf16 operands 1e-2 relative).  Cached vectors: the power iteration runs in
fp64 on both sides from the same stored inputs, and the new vector is
stored as fp32 (unit vector, rounding 6e-8): max abs difference 1e-6."""

import numpy as np
import pytest
import torch

from oracle import bjorck, checks, spectral
from paper_2601_13776_amd import orth
from paper_2601_13776_amd import workloads as wl

from gpu_util import DEV, to_dev, to_f64

pytestmark = pytest.mark.gpu

REL_F32 = 1e-5
BF16_REL = 1e-2
U_ABS = 1e-6


def stored(seed, shapes, dtype="f32"):
    w = wl.Workload("test", seed, dtype, 0, ())
    return [wl.stored_matrix(w, i, r, c) for i, (r, c) in enumerate(shapes)]


def cached(seed, shapes):
    rng = np.random.default_rng(seed)
    return [rng.standard_normal(min(s)).astype(np.float32) for s in shapes]


def run(st, us, iters, q, compute="f32"):
    ins = [to_dev(s) for s in st]
    outs = [torch.empty(t.shape, dtype=torch.float32, device=DEV) for t in ins]
    u = torch.from_numpy(np.concatenate(us)).to(DEV)
    status = torch.full((len(ins),), -1, dtype=torch.int32, device=DEV)
    orth.orth_orthogonalize_batched(ins, outs, iters, compute=compute, status=status, prescale="spectral",
                                    power_iters=q, u=u)
    torch.cuda.synchronize()
    u_new = u.cpu().numpy()
    offs = np.cumsum([0] + [len(x) for x in us])
    return outs, [u_new[offs[i]:offs[i + 1]] for i in range(len(us))], status.cpu().numpy()


SHAPES = [(1, 1), (1, 7), (7, 1), (16, 8), (8, 16), (33, 17), (64, 64), (128, 64), (64, 128), (100, 50),
          (65, 65), (129, 64), (200, 130), (256, 128), (128, 256), (300, 300), (512, 256)]


@pytest.mark.parametrize("q,iters", [(1, 12), (3, 8)])
def test_spectral_f32_mixed_batch(q, iters):
    st = stored(701, SHAPES)
    us = cached(702, SHAPES)
    outs, u_new, status = run(st, us, iters, q)
    assert np.all(status == 0)
    for s, u0, o, u1, shape in zip(st, us, outs, u_new, SHAPES):
        ref, v, _ = spectral.bjorck_spectral(s.astype(np.float64), u0.astype(np.float64), iters, q)
        assert checks.relative_difference(to_f64(o), ref) <= REL_F32, shape
        assert np.max(np.abs(u1 - v)) <= U_ABS, shape


@pytest.mark.parametrize("seed,q", [(0, 1), (1, 3)])
def test_spectral_random_ragged_batches(seed, q):
    """Seeded random ragged batches (1 to 600 rows and columns, tall and
    wide, fused and tiled) with 1 and 3 power steps, fp32 products."""
    rng = np.random.default_rng(800 + seed)
    shapes = [(int(rng.integers(1, 601)), int(rng.integers(1, 601))) for _ in range(5)] + \
             [(int(rng.integers(1, 129)), int(rng.integers(1, 65))) for _ in range(3)]
    print(f"[spectral random batch {seed}] q={q} {shapes}", flush=True)
    st = stored(810 + seed, shapes)
    us = cached(820 + seed, shapes)
    outs, u_new, status = run(st, us, 8, q)
    assert np.all(status == 0)
    for s, u0, o, u1, shape in zip(st, us, outs, u_new, shapes):
        ref, v, _ = spectral.bjorck_spectral(s.astype(np.float64), u0.astype(np.float64), 8, q)
        assert checks.relative_difference(to_f64(o), ref) <= REL_F32, shape
        assert np.max(np.abs(u1 - v)) <= U_ABS, shape


def test_spectral_bf16_batch():
    shapes = [(128, 64), (256, 128), (300, 700), (1024, 512), (512, 512), (2048, 1024)]
    st = stored(703, shapes, "bf16")
    us = cached(704, shapes)
    outs, u_new, status = run(st, us, 15, 2, compute="bf16")
    assert np.all(status == 0)
    for s, u0, o, u1, shape in zip(st, us, outs, u_new, shapes):
        ref, v, _ = spectral.bjorck_spectral(wl.as_f64(s), u0.astype(np.float64), 15, 2)
        assert checks.relative_difference(to_f64(o), ref) <= BF16_REL, shape
        assert checks.tile_relative_differences(to_f64(o), ref, 256).max() <= BF16_REL, shape
        assert np.max(np.abs(u1 - v)) <= U_ABS, shape


def test_spectral_cached_vector_reuse():
    """Two calls in a row: the second starts from the vectors the first
    wrote; with a cached top vector one power step suffices and rectangular
    matrices converge in fewer iterations than with Frobenius scaling."""
    shapes = [(256, 128), (96, 48), (1024, 512)]
    st = stored(705, shapes)
    us = cached(706, shapes)
    _, u1, _ = run(st, us, 10, 5)
    outs, u2, _ = run(st, [u.copy() for u in u1], 10, 1)
    for s, a, o, b, shape in zip(st, u1, outs, u2, shapes):
        ref, v, _ = spectral.bjorck_spectral(s.astype(np.float64), a.astype(np.float64), 10, 1)
        assert checks.relative_difference(to_f64(o), ref) <= REL_F32, shape
        assert np.max(np.abs(b - v)) <= U_ABS
        # 10 steps after spectral scaling reach orthogonality that Frobenius
        # scaling does not
        assert checks.gram_deviation(to_f64(o)) <= 1e-4, shape
        frob = bjorck.bjorck(s.astype(np.float64), 10)
        assert checks.gram_deviation(frob) > 10 * checks.gram_deviation(ref), shape


def test_spectral_statuses_and_zero_vector():
    shapes = [(40, 20), (40, 20), (20, 40), (300, 200), (70, 70)]
    st = stored(707, shapes)
    st[1] = np.zeros_like(st[1])
    st[2] = st[2].copy()
    st[2][1, 3] = np.inf
    us = cached(708, shapes)
    us[4] = np.zeros_like(us[4])       # a zero vector starts as ones
    outs, u_new, status = run(st, us, 6, 2)
    assert list(status) == [0, 1, 2, 0, 0]
    assert torch.all(outs[1] == 0) and torch.all(torch.isnan(outs[2]))
    assert np.array_equal(u_new[1], us[1]) and np.array_equal(u_new[2], us[2])
    for i in (0, 3, 4):
        ref, v, _ = spectral.bjorck_spectral(st[i].astype(np.float64), us[i].astype(np.float64), 6, 2)
        assert checks.relative_difference(to_f64(outs[i]), ref) <= REL_F32
        assert np.max(np.abs(u_new[i] - v)) <= U_ABS
