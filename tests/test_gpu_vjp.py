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
                  6e-2 square (about 2x the replayed error).  Each bound
                  holds for every 256 x 256 block as well as for the whole
                  matrix (the blocks measure within 1.1x of the whole), so
                  an error confined to a few blocks cannot hide in it.
"""

import numpy as np
import pytest
import torch

from oracle import bjorck_grad, checks
from paper_2601_13776_amd import orth
from paper_2601_13776_amd import workloads as wl

from gpu_util import DEV, random_geometries, to_dev, to_f64

pytestmark = pytest.mark.gpu

REL_F32 = 1e-5
REL_BF16_RECT = 1e-2
REL_BF16_SQUARE = 6e-2


def assert_bf16_close(got, ref, shape, what=""):
    """Whole-matrix and per-256-block relative difference within the bf16
    bound of the shape (square or rectangular)."""
    bound = REL_BF16_SQUARE if shape[0] == shape[1] else REL_BF16_RECT
    rel = checks.relative_difference(got, ref)
    blocks = checks.tile_relative_differences(got, ref, 256)
    assert rel <= bound, (shape, what, rel)
    assert blocks.max() <= bound, (shape, what, blocks.max(), np.unravel_index(np.argmax(blocks), blocks.shape))


def stored(seed, shapes, dtype="f32"):
    w = wl.Workload("test", seed, dtype, 0, ())
    return [wl.stored_matrix(w, i, r, c) for i, (r, c) in enumerate(shapes)]


def upstream(seed, shapes):
    """dL/d(output): N(0, 1) float32 matrices."""
    rng = np.random.default_rng(seed)
    return [rng.standard_normal(s).astype(np.float32) for s in shapes]


def run_vjp(st, gouts, iters, compute="f32", beta=0.5, prescale="frobenius", gin_dtype=None, tile=0):
    ws = [to_dev(s) for s in st]
    gos = [torch.from_numpy(g).to(DEV) for g in gouts]
    gis = [torch.empty(w.shape, dtype=w.dtype, device=DEV) for w in ws]
    status = torch.full((len(ws),), -1, dtype=torch.int32, device=DEV)
    orth.orth_orthogonalize_vjp_batched(ws, gos, gis, iters, beta=beta, prescale=prescale, compute=compute,
                                        status=status, tile=tile)
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


@pytest.mark.parametrize("tile", [0, 256])
def test_vjp_bf16_mixed_batch(tile):
    """bf16 parameters, fp32 upstream gradient, bf16 products (the small
    bucket runs in fp32 as in the forward); matrices with min(rows, cols)
    >= 1024 on the tile size chosen by occupancy or forced to 256."""
    print(f"[vjp bf16] mixed batch tile={tile}", flush=True)
    st = stored(205, SHAPES_BF16, "bf16")
    gouts = upstream(206, SHAPES_BF16)
    gis, status = run_vjp(st, gouts, 20, compute="bf16", tile=tile)
    assert np.all(status == 0)
    for s, g, o, shape in zip(st, gouts, gis, SHAPES_BF16):
        assert o.dtype == torch.bfloat16
        ref = bjorck_grad.bjorck_vjp(wl.as_f64(s), g.astype(np.float64), 20)
        assert_bf16_close(to_f64(o), ref, shape)


@pytest.mark.parametrize("beta,prescale,tile", [(0.25, "frobenius", 0), (0.5, "none", 256)])
def test_vjp_bf16_beta_and_no_prescale(beta, prescale, tile):
    """bf16 products with beta < 1/2, and without pre-scaling (inputs inside
    the basin), both tile classes and the small bucket."""
    shapes = [(128, 64), (256, 128), (512, 512), (1100, 1030)]
    st = stored(207, shapes)
    if prescale == "none":
        st = [(s / np.linalg.norm(s.astype(np.float64), 2) * 0.9).astype(np.float32) for s in st]
    gouts = upstream(208, shapes)
    gis, status = run_vjp(st, gouts, 12, compute="bf16", beta=beta, prescale=prescale, tile=tile)
    assert np.all(status == 0)
    for s, g, o, shape in zip(st, gouts, gis, shapes):
        ref = bjorck_grad.bjorck_vjp(s.astype(np.float64), g.astype(np.float64), 12, beta, prescale)
        assert_bf16_close(to_f64(o), ref, shape)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_vjp_random_ragged_batches(seed):
    """Seeded random ragged batches (1 to 600 rows and columns, tall and
    wide, fused and tiled) through the fp32 vector-Jacobian product."""
    rng = np.random.default_rng(700 + seed)
    shapes = [(int(rng.integers(1, 601)), int(rng.integers(1, 601))) for _ in range(5)] + \
             [(int(rng.integers(1, 129)), int(rng.integers(1, 65))) for _ in range(3)]
    print(f"[vjp random batch {seed}] {shapes}", flush=True)
    st = stored(710 + seed, shapes)
    gouts = upstream(720 + seed, shapes)
    gis, status = run_vjp(st, gouts, 6)
    assert np.all(status == 0)
    for s, g, o, shape in zip(st, gouts, gis, shapes):
        ref = bjorck_grad.bjorck_vjp(wl.as_f64(s), g.astype(np.float64), 6)
        assert checks.relative_difference(to_f64(o), ref) <= REL_F32, shape


def test_vjp_scale_invariance_property():
    """With Frobenius pre-scaling the gradient is orthogonal to W (any size)."""
    shapes = [(384, 200), (200, 384), (2048, 1024)]
    st = stored(207, shapes, "bf16")
    gouts = upstream(208, shapes)
    gis, _ = run_vjp(st, gouts, 15, compute="bf16", tile=256)
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


# ------------------------------------------------- composition VJP ---
from oracle import aoc, aoc_grad, bjorck  # noqa: E402

CONV_GEOMS = [(16, 16, 3, 1, 1, 1), (64, 128, 3, 2, 1, 1), (128, 512, 2, 2, 1, 1), (32, 32, 3, 1, 1, 4),
              (32, 32, 3, 1, 2, 1), (8, 8, 1, 1, 1, 1), (6, 6, 5, 2, 3, 3), (24, 16, 4, 2, 1, 2),
              (4, 6, 3, 1, 1, 1), (100, 70, 3, 1, 1, 1)]


def conv_factors(geom, seed, iters=40):
    rr, rc, npj, pr, pc = aoc.param_shapes(*geom)
    g = geom[5]
    rng = np.random.default_rng(seed)
    rko = np.stack([bjorck.bjorck(rng.standard_normal((rr, rc)), iters) for _ in range(g)]).astype(np.float32)
    proj = None
    if npj:
        proj = np.stack([np.stack([bjorck.bjorck(rng.standard_normal((pr, pc)), iters) for _ in range(npj)])
                         for _ in range(g)]).astype(np.float32)
    cin, cout, k = geom[0], geom[1], geom[2]
    dk = rng.standard_normal((cout, cin // g, k, k)).astype(np.float32)
    return rko, proj, dk


def conv_vjp_gpu(items, dtype=torch.float32):
    layers = []
    for geom, rko, proj, dk in items:
        t = lambda a: torch.from_numpy(a).to(DEV).to(dtype).contiguous()
        layers.append(dict(geom=geom, rko=t(rko), proj=t(proj) if proj is not None else None, grad_kernel=t(dk),
                           grad_rko=torch.full(rko.shape, float("nan"), dtype=dtype, device=DEV),
                           grad_proj=torch.full(proj.shape, float("nan"), dtype=dtype, device=DEV)
                           if proj is not None else None))
    orth.orth_build_conv_kernels_vjp_batched(layers)
    torch.cuda.synchronize()
    return layers


def test_conv_vjp_parity_batched():
    """Every geometry in one batched call (mixed k, stride, groups)."""
    items = [(geom, *conv_factors(geom, 300 + i)) for i, geom in enumerate(CONV_GEOMS)]
    layers = conv_vjp_gpu(items)
    for (geom, rko, proj, dk), L in zip(items, layers):
        ref_r, ref_p = aoc_grad.aoc_kernel_vjp(rko.astype(np.float64),
                                               None if proj is None else proj.astype(np.float64), *geom,
                                               dk.astype(np.float64))
        assert checks.relative_difference(to_f64(L["grad_rko"]), ref_r) <= REL_F32, geom
        if proj is not None:
            assert checks.relative_difference(to_f64(L["grad_proj"]), ref_p) <= REL_F32, geom


@pytest.mark.parametrize("geom", [(16, 16, 3, 1, 1, 1), (64, 128, 3, 2, 1, 1), (6, 6, 5, 2, 3, 3),
                                  (3, 64, 3, 1, 1, 1), (32, 64, 4, 2, 1, 1), (12, 12, 5, 1, 2, 2)])
def test_conv_vjp_parity_single(geom):
    rko, proj, dk = conv_factors(geom, 400)
    L = conv_vjp_gpu([(geom, rko, proj, dk)])[0]
    ref_r, ref_p = aoc_grad.aoc_kernel_vjp(rko.astype(np.float64), None if proj is None else proj.astype(np.float64),
                                           *geom, dk.astype(np.float64))
    assert checks.relative_difference(to_f64(L["grad_rko"]), ref_r) <= REL_F32
    if proj is not None:
        assert checks.relative_difference(to_f64(L["grad_proj"]), ref_p) <= REL_F32


def test_conv_vjp_random_geometries_batched():
    """Twelve seeded random geometries (groups, stride, dilation, k up to 5,
    ragged channel counts) in one batched call."""
    geoms = random_geometries(78, 12, aoc.param_shapes)
    print(f"[conv vjp random] {geoms}", flush=True)
    items = [(geom, *conv_factors(geom, 500 + i)) for i, geom in enumerate(geoms)]
    layers = conv_vjp_gpu(items)
    for (geom, rko, proj, dk), L in zip(items, layers):
        ref_r, ref_p = aoc_grad.aoc_kernel_vjp(rko.astype(np.float64),
                                               None if proj is None else proj.astype(np.float64), *geom,
                                               dk.astype(np.float64))
        assert checks.relative_difference(to_f64(L["grad_rko"]), ref_r) <= REL_F32, geom
        if proj is not None:
            assert checks.relative_difference(to_f64(L["grad_proj"]), ref_p) <= REL_F32, geom


def test_conv_vjp_bf16_storage():
    """bf16 storage of factors, kernel gradient and outputs (fp32 arithmetic):
    the oracle sees the bf16-rounded inputs; the outputs are rounded once
    (u = 2^-9), bound 1e-2."""
    geoms = [(64, 64, 3, 1, 1, 1), (32, 64, 4, 2, 1, 2)]
    items = []
    for i, geom in enumerate(geoms):
        rko, proj, dk = conv_factors(geom, 500 + i)
        r16 = lambda a: torch.from_numpy(a).to(torch.bfloat16).float().numpy()
        items.append((geom, r16(rko), r16(proj), r16(dk)))
    layers = conv_vjp_gpu(items, torch.bfloat16)
    for (geom, rko, proj, dk), L in zip(items, layers):
        ref_r, ref_p = aoc_grad.aoc_kernel_vjp(rko.astype(np.float64), proj.astype(np.float64), *geom,
                                               dk.astype(np.float64))
        assert checks.relative_difference(to_f64(L["grad_rko"]), ref_r) <= 1e-2
        assert checks.relative_difference(to_f64(L["grad_proj"]), ref_p) <= 1e-2


@pytest.mark.parametrize("compute,iters,tile", [("f32", 0, 0), ("f32", 7, 0), ("bf16", 6, 128), ("bf16", 6, 256)])
def test_saving_forward_and_saved_vjp(compute, iters, tile):
    """orth_orthogonalize_save_batched gives the forward's outputs and
    statuses; the VJP that takes its workspace (saved=True) gives the
    gradients of the recomputing VJP bit for bit, twice in a row (the saved
    iterates are left intact), including a zero matrix."""
    print(f"[saved vjp] compute={compute} iters={iters} tile={tile}", flush=True)
    shapes = [(16, 8), (8, 16), (100, 50), (300, 200), (200, 300), (256, 128), (1024, 1024), (40, 40)]
    st = stored(240, shapes, dtype="bf16" if compute == "bf16" else "f32")
    st[-1] = np.zeros_like(st[-1])
    gouts = upstream(241, shapes)
    ws = [to_dev(s) for s in st]
    ref_out = [torch.empty(w.shape, device=DEV) for w in ws]
    got_out = [torch.full(w.shape, float("nan"), device=DEV) for w in ws]
    st_ref = torch.full((len(ws),), -1, dtype=torch.int32, device=DEV)
    st_got = torch.full((len(ws),), -1, dtype=torch.int32, device=DEV)
    orth.orth_orthogonalize_batched(ws, ref_out, iters, compute=compute, status=st_ref, tile=tile)
    tape = orth.orth_orthogonalize_save_batched(ws, got_out, iters, compute=compute, status=st_got, tile=tile)
    gos = [torch.from_numpy(g).to(DEV) for g in gouts]
    g_ref = [torch.empty(w.shape, dtype=w.dtype, device=DEV) for w in ws]
    orth.orth_orthogonalize_vjp_batched(ws, gos, g_ref, iters, compute=compute, tile=tile)
    g_got = [[torch.full(w.shape, float("nan"), dtype=w.dtype, device=DEV) for w in ws] for _ in range(2)]
    st_vjp = torch.full((len(ws),), -1, dtype=torch.int32, device=DEV)
    for k, g in enumerate(g_got):
        orth.orth_orthogonalize_vjp_batched(ws, gos, g, iters, compute=compute, tile=tile, workspace=tape,
                                            saved=True, status=st_vjp if k else None)
    torch.cuda.synchronize()
    assert np.array_equal(st_got.cpu().numpy(), st_ref.cpu().numpy())
    assert np.array_equal(st_vjp.cpu().numpy(), st_ref.cpu().numpy())
    assert st_got.cpu().numpy()[-1] == 1
    for a, b, shape in zip(got_out[:-1], ref_out[:-1], shapes):
        # same arithmetic in both plans (tile lists differ only in order)
        assert checks.relative_difference(to_f64(a), to_f64(b)) <= 1e-6, shape
    assert torch.equal(got_out[-1], ref_out[-1]) and not torch.any(got_out[-1] != 0)
    for g in g_got:
        for a, b, shape in zip(g, g_ref, shapes):
            assert torch.equal(a, b), shape


def test_saving_forward_bf16_output_and_strides():
    """The saving forward writes bf16 outputs and honours leading dimensions
    (strided views) like the plain forward."""
    shapes = [(300, 200), (200, 300), (64, 48)]
    st = stored(242, shapes)
    ws = [to_dev(s) for s in st]
    big = [torch.full((r, c + 24), float("nan"), dtype=torch.bfloat16, device=DEV) for r, c in shapes]
    got = [b[:, 8:8 + c] for b, (r, c) in zip(big, shapes)]
    ref = [torch.empty(r, c, dtype=torch.bfloat16, device=DEV) for r, c in shapes]
    orth.orth_orthogonalize_batched(ws, ref, 6)
    orth.orth_orthogonalize_save_batched(ws, got, 6)
    torch.cuda.synchronize()
    for g, r, b, (rows, cols) in zip(got, ref, big, shapes):
        assert checks.relative_difference(to_f64(g), to_f64(r)) <= 1e-2 ** 2, (rows, cols)
        assert torch.all(torch.isnan(b[:, :8].float())) and torch.all(torch.isnan(b[:, 8 + cols:].float()))


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_saving_composition_and_saved_conv_vjp(dtype):
    """orth_build_conv_kernels_save_batched composes the kernels of
    orth_build_conv_kernels_batched; the composition VJP from its workspace
    (saved=True) equals the recomputing one bit for bit, twice in a row."""
    print(f"[saved conv vjp] {dtype}", flush=True)
    items = [(geom, *conv_factors(geom, 600 + i)) for i, geom in enumerate(CONV_GEOMS)]
    t = lambda a: torch.from_numpy(a).to(DEV).to(dtype).contiguous()
    fwd_ref, fwd_got = [], []
    for geom, rko, proj, dk in items:
        cin, cout, k = geom[0], geom[1], geom[2]
        shape = (cout, cin // geom[5], k, k)
        fwd_ref.append(dict(geom=geom, rko=t(rko), proj=t(proj) if proj is not None else None,
                            kernel=torch.empty(shape, dtype=dtype, device=DEV)))
        fwd_got.append(dict(geom=geom, rko=fwd_ref[-1]["rko"], proj=fwd_ref[-1]["proj"],
                            kernel=torch.full(shape, float("nan"), dtype=dtype, device=DEV)))
    orth.orth_build_conv_kernels_batched(fwd_ref)
    tape = orth.orth_build_conv_kernels_save_batched(fwd_got)
    ref = conv_vjp_gpu(items, dtype)
    got = []
    for _ in range(2):
        layers = []
        for (geom, rko, proj, dk), F in zip(items, fwd_got):
            layers.append(dict(geom=geom, rko=F["rko"], proj=F["proj"], grad_kernel=t(dk),
                               grad_rko=torch.full(rko.shape, float("nan"), dtype=dtype, device=DEV),
                               grad_proj=torch.full(proj.shape, float("nan"), dtype=dtype, device=DEV)
                               if proj is not None else None))
        orth.orth_build_conv_kernels_vjp_batched(layers, workspace=tape, saved=True)
        got.append(layers)
    torch.cuda.synchronize()
    for a, b, (geom, *_) in zip(fwd_got, fwd_ref, items):
        tol = 1e-6 if dtype == torch.float32 else 1e-2
        assert checks.relative_difference(to_f64(a["kernel"]), to_f64(b["kernel"])) <= tol, geom
    for layers in got:
        for L, R, (geom, *_) in zip(layers, ref, items):
            assert torch.equal(L["grad_rko"], R["grad_rko"]), geom
            if R["grad_proj"] is not None:
                assert torch.equal(L["grad_proj"], R["grad_proj"]), geom


def test_layer_vjp_chain():
    """Raw parameters -> kernel gradient -> raw-parameter gradients, all on
    the GPU (Björck forward, composition VJP, Björck VJP), against the
    oracle's whole-layer VJP."""
    geom, iters = (32, 32, 3, 1, 1, 2), 15
    cin, cout, k, s, d, g = geom
    rr, rc, npj, pr, pc = aoc.param_shapes(*geom)
    rng = np.random.default_rng(600)
    raw_rko = rng.standard_normal((g, rr, rc)).astype(np.float32)
    raw_proj = rng.standard_normal((g, npj, pr, pc)).astype(np.float32)
    dk = rng.standard_normal((cout, cin // g, k, k)).astype(np.float32)
    raws = [torch.from_numpy(m).to(DEV) for m in list(raw_rko) + list(raw_proj.reshape(-1, pr, pc))]
    outs = [torch.empty_like(t) for t in raws]
    orth.orth_orthogonalize_batched(raws, outs, iters)
    rko = torch.stack(outs[:g]).contiguous()
    proj = torch.stack(outs[g:]).reshape(g, npj, pr, pc).contiguous()
    L = dict(geom=geom, rko=rko, proj=proj, grad_kernel=torch.from_numpy(dk).to(DEV),
             grad_rko=torch.empty_like(rko), grad_proj=torch.empty_like(proj))
    orth.orth_build_conv_kernels_vjp_batched([L])
    gouts = list(L["grad_rko"]) + list(L["grad_proj"].reshape(-1, pr, pc))
    gins = [torch.empty_like(t) for t in raws]
    orth.orth_orthogonalize_vjp_batched(raws, [t.contiguous() for t in gouts], gins, iters)
    torch.cuda.synchronize()
    ref_r, ref_p = aoc_grad.aoc_layer_vjp(raw_rko.astype(np.float64), raw_proj.astype(np.float64), *geom, iters,
                                          dk.astype(np.float64))
    got_r = np.stack([to_f64(t) for t in gins[:g]])
    got_p = np.stack([to_f64(t) for t in gins[g:]]).reshape(ref_p.shape)
    assert checks.relative_difference(got_r, ref_r) <= REL_F32
    assert checks.relative_difference(got_p, ref_p) <= REL_F32


# ------------------------------------------- spectral pre-scaling (f1 x f2) --

def cached_vectors(seed, shapes):
    rng = np.random.default_rng(seed)
    return [rng.standard_normal(min(s)).astype(np.float32) for s in shapes]


def spectral_vjp(st, gouts, us, iters, q, compute="f32", tile=0):
    ws = [to_dev(s) for s in st]
    gos = [torch.from_numpy(g).to(DEV) for g in gouts]
    gis = [torch.empty(w.shape, dtype=w.dtype, device=DEV) for w in ws]
    u = torch.from_numpy(np.concatenate(us)).to(DEV)
    u_before = u.clone()
    status = torch.full((len(ws),), -1, dtype=torch.int32, device=DEV)
    orth.orth_orthogonalize_vjp_batched(ws, gos, gis, iters, compute=compute, status=status, tile=tile,
                                        prescale="spectral", power_iters=q, u=u)
    torch.cuda.synchronize()
    assert torch.equal(u, u_before), "the vector-Jacobian product must not write the cached vectors"
    return gis, status.cpu().numpy()


SPEC_SHAPES_F32 = [(16, 8), (8, 16), (40, 40), (128, 64), (100, 50), (65, 65), (200, 130), (130, 300), (512, 256)]


@pytest.mark.parametrize("q", [1, 3])
def test_vjp_spectral_f32_mixed_batch(q):
    """Spectral pre-scaling from cached vectors (held constant) through q
    power steps: small (fused kernel) and tiled matrices, tall and wide,
    against oracle.spectral.bjorck_spectral_vjp."""
    from oracle import spectral
    print(f"[vjp spectral f32] q={q}", flush=True)
    st = stored(221, SPEC_SHAPES_F32)
    gouts = upstream(222, SPEC_SHAPES_F32)
    us = cached_vectors(223, SPEC_SHAPES_F32)
    gis, status = spectral_vjp(st, gouts, us, 8, q)
    assert np.all(status == 0)
    for s, g, u, o, shape in zip(st, gouts, us, gis, SPEC_SHAPES_F32):
        ref = spectral.bjorck_spectral_vjp(wl.as_f64(s), u.astype(np.float64), g.astype(np.float64), 8, q)
        rel = checks.relative_difference(to_f64(o), ref)
        assert rel <= REL_F32, (shape, q, rel)


def test_vjp_spectral_floor_branch():
    """Cached vectors on a small singular direction: the power estimate stays
    below ||W||_F / sqrt(N), the floor sets the scale and its derivative
    applies (fused and tiled matrices).  Singular values near 1.5 and 1
    keep the largest one of W_0 below sqrt(3) under the floor's scale."""
    from oracle import spectral
    rng = np.random.default_rng(224)
    shapes = [(48, 40), (200, 130)]
    st, us = [], []
    for r, c in shapes:
        w = 0.001 * rng.standard_normal((r, c))
        w[np.arange(c), np.arange(c)] += 1.0
        w[0, 0] = 1.5
        st.append(w.astype(np.float32))
        u = np.zeros(c, dtype=np.float32)
        u[1] = 1.0
        us.append(u)
    gouts = upstream(225, shapes)
    for s, u in zip(st, us):
        _, _, sigma, _ = spectral.spectral_prescale(s.astype(np.float64), u.astype(np.float64), 1)
        floor = np.sqrt(np.sum(s.astype(np.float64) ** 2)) / np.sqrt(min(s.shape))
        assert abs(sigma - floor) <= 1e-12 * floor
    gis, status = spectral_vjp(st, gouts, us, 6, 1)
    assert np.all(status == 0)
    for s, g, u, o in zip(st, gouts, us, gis):
        ref = spectral.bjorck_spectral_vjp(s.astype(np.float64), u.astype(np.float64), g.astype(np.float64), 6, 1)
        assert checks.relative_difference(to_f64(o), ref) <= REL_F32, s.shape


SPEC_SHAPES_BF16 = [(128, 64), (64, 100), (256, 128), (300, 700), (1024, 512), (512, 512)]


@pytest.mark.parametrize("q", [1, 2])
def test_vjp_spectral_bf16_mixed_batch(q):
    from oracle import spectral
    print(f"[vjp spectral bf16] q={q}", flush=True)
    st = stored(226, SPEC_SHAPES_BF16, "bf16")
    gouts = upstream(227, SPEC_SHAPES_BF16)
    us = cached_vectors(228, SPEC_SHAPES_BF16)
    gis, status = spectral_vjp(st, gouts, us, 20, q, compute="bf16")
    assert np.all(status == 0)
    for s, g, u, o, shape in zip(st, gouts, us, gis, SPEC_SHAPES_BF16):
        ref = spectral.bjorck_spectral_vjp(wl.as_f64(s), u.astype(np.float64), g.astype(np.float64), 20, q)
        assert_bf16_close(to_f64(o), ref, shape, f"q={q}")


def test_vjp_spectral_saved_and_statuses():
    """The training pattern with spectral pre-scaling: the saving forward
    gives the outputs and new cached vectors of orth_orthogonalize_batched,
    and the VJP from its workspace (no cached vectors passed) equals the
    recomputing VJP given the vectors the forward started from, bit for
    bit; a zero matrix gets a zero gradient."""
    shapes = [(40, 20), (96, 96), (300, 200), (130, 64)]
    st = stored(229, shapes)
    st[1][:] = 0
    ins = [to_dev(s) for s in st]
    us = cached_vectors(230, shapes)
    u0 = torch.from_numpy(np.concatenate(us)).to(DEV)
    gouts = [torch.from_numpy(g).to(DEV) for g in upstream(231, shapes)]
    # plain forward
    u_a = u0.clone()
    outs_a = [torch.empty(s, device=DEV) for s in shapes]
    orth.orth_orthogonalize_batched(ins, outs_a, 7, prescale="spectral", power_iters=2, u=u_a)
    # saving forward, then the saved VJP
    u_b = u0.clone()
    outs_b = [torch.empty(s, device=DEV) for s in shapes]
    status = torch.full((len(shapes),), -1, dtype=torch.int32, device=DEV)
    tape = orth.orth_orthogonalize_save_batched(ins, outs_b, 7, prescale="spectral", power_iters=2, u=u_b,
                                                status=status)
    g_saved = [torch.empty_like(t) for t in ins]
    orth.orth_orthogonalize_vjp_batched(ins, gouts, g_saved, 7, prescale="spectral", power_iters=2,
                                        workspace=tape, saved=True)
    # recomputing VJP from the vectors the forward started from
    g_rec = [torch.empty_like(t) for t in ins]
    orth.orth_orthogonalize_vjp_batched(ins, gouts, g_rec, 7, prescale="spectral", power_iters=2, u=u0.clone())
    torch.cuda.synchronize()
    assert list(status.cpu().numpy()) == [0, 1, 0, 0]
    # same arithmetic in both plans (tile lists differ only in order)
    assert torch.allclose(u_a, u_b, rtol=1e-6, atol=1e-7)
    for a, b, shape in zip(outs_a, outs_b, shapes):
        assert checks.relative_difference(to_f64(a), to_f64(b)) <= 1e-6, shape
    for a, b in zip(g_saved, g_rec):
        assert torch.equal(a, b)
    assert bool((g_rec[1] == 0).all())
