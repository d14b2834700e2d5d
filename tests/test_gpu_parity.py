"""GPU parity: the HIP path (through the C ABI) against the float64 oracle on
the same seeded inputs.

Tolerances (stated by the target):
  fp32 compute : relative Frobenius difference to the oracle <= 1e-5;
                 max |W^T W - I| <= 1e-5 for matrices that have converged.
  bf16 operands, fp32 accumulation : max |W^T W - I| <= 3e-3 for converged
                 matrices.  Element-wise, rounding the product operands to
                 bf16 (unit roundoff u = 2^-9) moves the iterate by a few u in
                 relative Frobenius norm: BF16_REL = 1e-2 (about 5 u) for
                 every matrix, converged or not.
"""

import math
import os

import numpy as np
import pytest
import torch

from oracle import aoc, bjorck, checks, conv
from paper_2601_13776_amd import orth
from paper_2601_13776_amd import workloads as wl

from gpu_util import DEV, gpu_orthogonalize, oracle_inputs, random_geometries, to_dev, to_f64

pytestmark = pytest.mark.gpu

REL_F32 = 1e-5
ORTH_F32 = 1e-5
ORTH_BF16 = 3e-3
BF16_REL = 1e-2


def stored(seed, shapes, dtype="f32"):
    w = wl.Workload("test", seed, dtype, 0, ())
    return [wl.stored_matrix(w, i, r, c) for i, (r, c) in enumerate(shapes)]


def t_conv(mats64, tol=1e-6):
    return max(bjorck.iterations_to_converge(m, tol=tol) for m in mats64) + 2


def converged_at(m64, iters, tol=1e-6):
    return bjorck.iterations_to_converge(m64, tol=tol) <= iters


# ---------------------------------------------------------------- Björck --

SMALL = [(1, 1), (1, 7), (7, 1), (16, 8), (8, 16), (16, 16), (33, 17), (64, 64), (128, 64), (64, 128),
         (100, 50), (31, 64), (128, 33), (32, 32)]
TILED_F32 = [(65, 65), (129, 64), (200, 130), (256, 128), (128, 256), (300, 300), (512, 256), (1024, 512)]


@pytest.mark.parametrize("iters", [0, 1, 12])
def test_f32_mixed_batch(iters):
    """One batched call over small (fused LDS kernel) and tiled matrices,
    ragged shapes, tall and wide."""
    shapes = SMALL + TILED_F32
    st = stored(101, shapes)
    outs, status = gpu_orthogonalize(st, iters)
    assert np.all(status == 0)
    for s, o, shape in zip(oracle_inputs(st), outs, shapes):
        ref = bjorck.bjorck(s, iters)
        got = to_f64(o)
        assert got.shape == shape
        rel = checks.relative_difference(got, ref)
        assert rel <= REL_F32, (shape, rel)


def test_f32_converged_orthogonality():
    shapes = [(16, 16), (16, 8), (64, 64), (64, 32), (256, 128), (128, 256), (300, 300)]
    st = stored(102, shapes)
    x64 = oracle_inputs(st)
    iters = t_conv(x64)
    outs, _ = gpu_orthogonalize(st, iters)
    for s, o, shape in zip(x64, outs, shapes):
        got = to_f64(o)
        assert checks.gram_deviation(got) <= ORTH_F32, shape
        assert checks.relative_difference(got, bjorck.bjorck(s, iters)) <= REL_F32, shape


@pytest.mark.parametrize("beta", [0.5, 0.25])
def test_beta_and_no_prescale(beta):
    shapes = [(40, 20), (300, 200)]
    st = stored(103, shapes)
    x64 = oracle_inputs(st)
    # inputs already scaled so that no pre-scaling is needed
    pre = [(x / np.linalg.norm(x)).astype(np.float32) for x in x64]
    outs, _ = gpu_orthogonalize(pre, 7, beta=beta, prescale="none")
    for p, o in zip(pre, outs):
        ref = bjorck.bjorck(p.astype(np.float64), 7, beta=beta, prescale="none")
        assert checks.relative_difference(to_f64(o), ref) <= REL_F32


@pytest.mark.parametrize("beta,tile", [(0.25, 0), (0.25, 256), (0.5, 128)])
def test_bf16_beta_and_no_prescale(beta, tile):
    """bf16 products with beta < 1/2 and without pre-scaling (the caller's
    scale is the iterate's start), on both tile classes and the fused
    small-matrix kernel."""
    shapes = [(40, 20), (256, 128), (1024, 1024), (1100, 1030)]
    st = stored(113, shapes)
    pre = [(x / np.linalg.norm(x)).astype(np.float32) for x in oracle_inputs(st)]
    outs, status = gpu_orthogonalize(pre, 12, compute="bf16", beta=beta, prescale="none", tile=tile)
    assert np.all(status == 0)
    for p, o, shape in zip(pre, outs, shapes):
        ref = bjorck.bjorck(p.astype(np.float64), 12, beta=beta, prescale="none")
        got = to_f64(o)
        assert checks.relative_difference(got, ref) <= BF16_REL, shape
        assert checks.tile_relative_differences(got, ref, 256).max() <= BF16_REL, shape


BF16_SHAPES = [(256, 128), (128, 256), (384, 200), (1024, 512), (2048, 1000), (1000, 2048), (1024, 1024),
               (1100, 1030), (64, 32), (32, 32)]


@pytest.mark.parametrize("tile", [0, 128, 256])
def test_bf16_mixed_batch(tile):
    """Every size class; the matrices with min(rows, cols) >= 1024 run on
    the tile size chosen by occupancy (0) or forced to 128 / 256."""
    print(f"[bf16 mixed] tile={tile}", flush=True)
    st = stored(104, BF16_SHAPES, dtype="bf16")
    x64 = oracle_inputs(st)
    iters = 20
    outs, status = gpu_orthogonalize(st, iters, compute="bf16", tile=tile)
    assert np.all(status == 0)
    for s, o, shape in zip(x64, outs, BF16_SHAPES):
        ref = bjorck.bjorck(s, iters)
        got = to_f64(o)
        rel = checks.relative_difference(got, ref)
        assert rel <= BF16_REL, (shape, rel)
        if converged_at(s, iters):
            assert checks.gram_deviation(got) <= ORTH_BF16, shape
        else:
            # not converged: the deviation from orthogonality is the oracle's
            assert abs(checks.gram_deviation(got) - checks.gram_deviation(ref)) <= ORTH_BF16, shape


def test_bf16_two_tile_classes_and_timing_span():
    """A batch with both bf16 tile classes (the N >= 1024 matrices forced to
    256-tiles): the same bits as each class's matrices orthogonalized in
    calls of their own, the oracle's result on a sampled large matrix, and
    a timing span (the union of the launches' intervals) between the longer
    class's kernel time and the sum of both."""
    shapes = [(2048, 2048)] * 4 + [(512, 256), (256, 512), (384, 384), (1000, 130)] * 2 + [(32, 32), (64, 48)] * 3
    st = stored(109, shapes, dtype="bf16")
    ins = [to_dev(a) for a in st]
    iters = 6
    print("[bf16 two classes] combined call", flush=True)
    orth.orth_timing_enable(True)
    orth.orth_timing_reset()
    both = [torch.empty(t.shape, device=DEV) for t in ins]
    orth.orth_orthogonalize_batched(ins, both, iters, compute="bf16", tile=256)
    torch.cuda.synchronize()
    t256, n256 = orth.orth_timing_read("bjorck_bf16_256")
    t128, n128 = orth.orth_timing_read("bjorck_bf16_128")
    span, n = orth.orth_timing_span("bjorck_bf16_")
    tsmall, nsmall = orth.orth_timing_read("bjorck_small")
    span_all, n_all = orth.orth_timing_span("bjorck_")
    orth.orth_timing_enable(False)
    orth.orth_timing_reset()
    assert n256 == n128 == 2 * iters and n == n256 + n128
    assert max(t256, t128) * 0.999 <= span <= (t256 + t128) * 1.001
    # the small matrices' kernels run on side streams beside the tiled ones
    assert nsmall >= 1 and n_all == n + nsmall
    assert span * 0.999 <= span_all <= (span + tsmall) * 1.001
    print("[bf16 two classes] classes apart", flush=True)
    for part in ([0, 1, 2, 3], list(range(4, len(shapes)))):
        outs = [torch.empty(ins[i].shape, device=DEV) for i in part]
        orth.orth_orthogonalize_batched([ins[i] for i in part], outs, iters, compute="bf16", tile=256)
        torch.cuda.synchronize()
        for i, o in zip(part, outs):
            assert torch.equal(o, both[i]), shapes[i]
    ref = bjorck.bjorck(oracle_inputs([st[3]])[0], iters)
    assert checks.relative_difference(to_f64(both[3]), ref) <= BF16_REL
    assert checks.tile_relative_differences(to_f64(both[3]), ref, 256).max() <= BF16_REL


@pytest.mark.parametrize("seed", [0, 1, 2, 3, 4])
def test_random_ragged_batches(seed):
    """Seeded random batches of ragged shapes (1 to 1100 rows and columns,
    tall and wide, every size class) through both product precisions,
    against the oracle whole and per 256-block."""
    rng = np.random.default_rng(900 + seed)
    shapes = [(int(rng.integers(1, 1101)), int(rng.integers(1, 1101))) for _ in range(6)] + \
             [(int(rng.integers(1, 129)), int(rng.integers(1, 65))) for _ in range(4)]
    print(f"[random batch {seed}] {shapes}", flush=True)
    for compute, dtype, bound in (("f32", "f32", REL_F32), ("bf16", "bf16", BF16_REL)):
        st = stored(950 + seed, shapes, dtype=dtype)
        outs, status = gpu_orthogonalize(st, 8, compute=compute)
        assert np.all(status == 0)
        for s, o, shape in zip(oracle_inputs(st), outs, shapes):
            ref = bjorck.bjorck(s, 8)
            got = to_f64(o)
            assert checks.relative_difference(got, ref) <= bound, (compute, shape)
            if compute == "bf16" and min(shape) > 1:
                assert checks.tile_relative_differences(got, ref, 256).max() <= bound, (compute, shape)


# K-loop lengths of the bf16 tile kernel: with 64-deep k-steps, a Gram tile
# runs Mp / 64 k-steps and an update tile tj * T / 64 (stored-tile part)
# plus (Np - tj * T) / 64 (the rest) for tile size T, always even; the loop
# runs whole six-step periods and a remainder of 0, 2 or 4 k-steps, each a
# different stretch of straight-line code with its own buffer rotation and
# wait counts.  These shapes give every remainder in each kind of loop, for
# both tile sizes, and the results are checked whole and per block.
KLOOP_SHAPES = {256: [(1536, 1024), (1280, 1280), (1024, 1024), (1024, 1792)],
                128: [(384, 200), (256, 128), (512, 256), (640, 384), (768, 768)]}


@pytest.mark.parametrize("tile", [128, 256])
def test_bf16_k_loop_remainders(tile):
    shapes = KLOOP_SHAPES[tile]
    print(f"[bf16 k-loop remainders] tile={tile} shapes={shapes}", flush=True)
    for m, n in shapes:   # the shapes above do span every remainder
        mp, np_ = -(-max(m, n) // tile) * tile, -(-min(m, n) // tile) * tile
        assert min(m, n) > 64 and (tile == 128 or min(m, n) >= 1024)
        assert (mp // 64) % 2 == 0 and (np_ // 64) % 2 == 0
    gram = {(-(-max(m, n) // tile) * tile // 64) % 6 for m, n in shapes}
    upd = set()
    for m, n in shapes:
        np_ = -(-min(m, n) // tile) * tile
        for tj in range(np_ // tile):
            upd |= {(tj * tile // 64) % 6, ((np_ - tj * tile) // 64) % 6}
    assert gram == {0, 2, 4} and upd == {0, 2, 4}, (gram, upd)
    st = stored(131 + tile, shapes, dtype="bf16")
    x64 = oracle_inputs(st)
    iters = 8
    outs, status = gpu_orthogonalize(st, iters, compute="bf16", tile=tile)
    assert np.all(status == 0)
    for s, o, shape in zip(x64, outs, shapes):
        ref = bjorck.bjorck(s, iters)
        got = to_f64(o)
        assert checks.relative_difference(got, ref) <= BF16_REL, shape
        tiles = checks.tile_relative_differences(got, ref, tile)
        assert tiles.max() <= BF16_REL, (shape, tiles.max(), np.unravel_index(np.argmax(tiles), tiles.shape))


def test_concurrent_calls_two_threads():
    """Two host threads, each on a stream of its own, run mixed batches
    (small matrices on the library's side streams, tiled ones on the
    caller's stream) at the same time, three calls each; every result is
    bit-identical to the same call made alone, which matches the oracle."""
    import threading

    print("[concurrent] two threads x 3 calls", flush=True)
    jobs = [(stored(111, SMALL + TILED_F32), "f32", 12),
            (stored(112, [(256, 128), (384, 200), (1024, 512), (64, 32), (32, 32), (100, 50)], dtype="bf16"),
             "bf16", 20)]
    alone = []
    for st_list, comp, iters in jobs:
        outs, status = gpu_orthogonalize(st_list, iters, compute=comp)
        assert np.all(status == 0)
        alone.append([o.clone() for o in outs])
    # the fp32 batch made alone against the oracle
    for s, o in zip(oracle_inputs(jobs[0][0]), alone[0]):
        assert checks.relative_difference(to_f64(o), bjorck.bjorck(s, 12)) <= REL_F32
    ins = [[to_dev(s) for s in st_list] for st_list, _, _ in jobs]
    results = [[None] * 3 for _ in jobs]
    errors = []
    torch.cuda.synchronize()

    def run(j):
        try:
            stream = torch.cuda.Stream()
            _, comp, iters = jobs[j]
            with torch.cuda.stream(stream):
                for rep in range(3):
                    outs = [torch.empty(t.shape, dtype=torch.float32, device=DEV) for t in ins[j]]
                    status = torch.full((len(outs),), -1, dtype=torch.int32, device=DEV)
                    orth.orth_orthogonalize_batched(ins[j], outs, iters, compute=comp, status=status)
                    results[j][rep] = (outs, status)
            stream.synchronize()
        except Exception as e:  # re-raised by the main thread
            errors.append(e)

    threads = [threading.Thread(target=run, args=(j,)) for j in range(len(jobs))]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    torch.cuda.synchronize()
    assert not errors, errors
    for j in range(len(jobs)):
        for rep in range(3):
            outs, status = results[j][rep]
            assert np.all(status.cpu().numpy() == 0), (j, rep)
            for a, b in zip(alone[j], outs):
                assert torch.equal(a, b), (j, rep, tuple(a.shape))


@pytest.mark.parametrize("tile", [0, 256])
def test_bf16_converged_all(tile):
    shapes = [(256, 256), (1024, 1024), (512, 256)]
    st = stored(105, shapes, dtype="bf16")
    x64 = oracle_inputs(st)
    iters = t_conv(x64)
    outs, _ = gpu_orthogonalize(st, iters, compute="bf16", tile=tile)
    for o, shape in zip(outs, shapes):
        assert checks.gram_deviation(to_f64(o)) <= ORTH_BF16, shape


# ------------------------------------------------------------ edge cases --

def test_empty_batch():
    orth.orth_orthogonalize_batched([], [], 5)


@pytest.mark.filterwarnings("ignore:The CUDA Graph is empty")
def test_calls_refuse_stream_capture():
    """Calls that copy descriptor tables refuse a capturing stream before
    enqueuing anything (a captured copy would read a staging buffer that
    later calls refill); the stream works normally afterwards."""
    st = stored(110, [(300, 200), (40, 20)])
    ins = [to_dev(a) for a in st]
    outs = [torch.empty(t.shape, device=DEV) for t in ins]
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with pytest.raises(orth.OrthError) as e:
        with torch.cuda.graph(g):
            orth.orth_orthogonalize_batched(ins, outs, 5)
    assert e.value.code == orth.ORTH_EUNSUPPORTED and "captured" in str(e.value)
    torch.cuda.synchronize()
    got, status = gpu_orthogonalize(st, 5)
    assert np.all(status == 0)
    for s, o in zip(oracle_inputs(st), got):
        assert checks.relative_difference(to_f64(o), bjorck.bjorck(s, 5)) <= REL_F32


@pytest.mark.parametrize("shape", [(16, 8), (300, 200)])
def test_zero_and_nonfinite(shape):
    z = np.zeros(shape, dtype=np.float32)
    n = np.ones(shape, dtype=np.float32)
    n[3, 2] = np.nan
    good = stored(106, [shape])[0]
    outs, status = gpu_orthogonalize([z, n, good], 5)
    assert list(status) == [1, 2, 0]
    assert torch.all(outs[0] == 0)
    assert torch.all(torch.isnan(outs[1]))
    assert checks.relative_difference(to_f64(outs[2]), bjorck.bjorck(good.astype(np.float64), 5)) <= REL_F32


@pytest.mark.parametrize("shape", [(20, 12), (260, 130)])
def test_inplace_strided_and_bf16_out(shape):
    st = stored(107, [shape])[0]
    ref = bjorck.bjorck(st.astype(np.float64), 9)
    # in place
    t = to_dev(st)
    orth.orth_orthogonalize_batched([t], [t], 9)
    torch.cuda.synchronize()
    assert checks.relative_difference(to_f64(t), ref) <= REL_F32
    # leading dimension larger than cols, both sides
    big_in = torch.zeros(shape[0], shape[1] + 5, device=DEV)
    big_in[:, :shape[1]] = to_dev(st)
    big_out = torch.full((shape[0], shape[1] + 3), 7.0, device=DEV)
    orth.orth_orthogonalize_batched([big_in[:, :shape[1]]], [big_out[:, :shape[1]]], 9)
    torch.cuda.synchronize()
    assert checks.relative_difference(to_f64(big_out[:, :shape[1]]), ref) <= REL_F32
    assert torch.all(big_out[:, shape[1]:] == 7.0)
    # bf16 output (rounded once from the fp32 iterate)
    o = torch.empty(shape, dtype=torch.bfloat16, device=DEV)
    orth.orth_orthogonalize_batched([to_dev(st)], [o], 9)
    torch.cuda.synchronize()
    assert checks.relative_difference(to_f64(o), ref) <= 4e-3


@pytest.mark.parametrize("compute,shape,iters", [("f32", (256, 128), 0), ("f32", (256, 128), 5),
                                                 ("f32", (512, 256), 6), ("bf16", (1024, 1024), 5),
                                                 ("bf16", (1024, 512), 0)])
def test_output_holding_the_iterate(compute, shape, iters):
    """fp32 outputs laid out as the fp32 iterate (no padding, ld_out = cols)
    hold the iterate during the call: the same bits as an output with a
    wider row stride (which keeps the workspace buffer and the write-out
    pass), also in place, and zero or non-finite inputs still give zeros or
    NaN there."""
    st = stored(108, [shape] * 3)
    st[1][:] = 0.0
    st[2][5, 3] = np.nan
    ins = [to_dev(a) for a in st]
    if compute == "bf16":
        ins = [t.to(torch.bfloat16) for t in ins]
    plain = [torch.full(shape, 3.0, device=DEV) for _ in ins]
    wide = [torch.full((shape[0], shape[1] + 8), 3.0, device=DEV) for _ in ins]
    views = [w[:, :shape[1]] for w in wide]
    for outs in (plain, views):
        status = torch.zeros(3, dtype=torch.int32, device=DEV)
        orth.orth_orthogonalize_batched(ins, outs, iters, compute=compute, status=status)
        torch.cuda.synchronize()
        assert status.tolist() == [0, 1, 2]
    for a, b in zip(plain, views):
        assert torch.equal(a, b) or (torch.isnan(a).all() and torch.isnan(b).all())
    assert torch.all(plain[1] == 0) and torch.all(torch.isnan(plain[2]))
    assert torch.all(wide[0][:, shape[1]:] == 3.0)
    ref = bjorck.bjorck(to_f64(ins[0]), iters)
    assert checks.relative_difference(to_f64(plain[0]), ref) <= (REL_F32 if compute == "f32" else BF16_REL)
    # in place (fp32 input and output)
    t = to_dev(st[0])
    orth.orth_orthogonalize_batched([t], [t], iters, compute=compute)
    torch.cuda.synchronize()
    if compute == "f32":
        assert torch.equal(t, plain[0])
    else:   # the bf16 copies now round the fp32 input, not a bf16 one
        assert checks.relative_difference(to_f64(t), bjorck.bjorck(st[0].astype(np.float64), iters)) <= BF16_REL


# ------------------------------------------------------------ composition --

COMPOSE_GEOMS = [(16, 16, 3, 1, 1, 1), (64, 128, 3, 2, 1, 1), (128, 512, 2, 2, 1, 1), (32, 32, 3, 1, 1, 4),
                 (32, 32, 3, 1, 2, 1), (8, 8, 1, 1, 1, 1), (6, 6, 5, 2, 3, 3), (24, 16, 4, 2, 1, 2),
                 (4, 6, 3, 1, 1, 1), (100, 70, 3, 1, 1, 1),
                 # a 3-channel stem and head (rank-1 projectors on 3 channels), k = 7,
                 # even k with stride, dilation with groups, k = s with groups
                 (3, 64, 3, 1, 1, 1), (64, 3, 3, 1, 1, 1), (64, 64, 7, 1, 1, 1), (32, 64, 4, 2, 1, 1),
                 (48, 48, 3, 1, 2, 3), (16, 32, 2, 2, 1, 2), (12, 12, 5, 1, 2, 2)]


def oracle_factors(geom, seed, iters=40):
    rr, rc, npj, pr, pc = aoc.param_shapes(*geom)
    g = geom[5]
    rng = np.random.default_rng(seed)
    rko = np.stack([bjorck.bjorck(rng.standard_normal((rr, rc)), iters) for _ in range(g)]).astype(np.float32)
    proj = None
    if npj:
        proj = np.stack([np.stack([bjorck.bjorck(rng.standard_normal((pr, pc)), iters) for _ in range(npj)])
                         for _ in range(g)]).astype(np.float32)
    return rko, proj


@pytest.mark.parametrize("geom", COMPOSE_GEOMS)
def test_compose_parity(geom):
    """GPU composition of given fp32 factors vs the oracle's composition of
    the same factors."""
    cin, cout, k, s, d, g = geom
    rko, proj = oracle_factors(geom, sum(geom))
    kern = torch.empty(cout, cin // g, k, k, device=DEV)
    orth.orth_build_conv_kernel(to_dev(rko), to_dev(proj) if proj is not None else None, cin, cout, k, s, d, g,
                                kern)
    torch.cuda.synchronize()
    ref = aoc.aoc_kernel(rko.astype(np.float64), None if proj is None else proj.astype(np.float64), *geom)
    assert checks.relative_difference(to_f64(kern), ref) <= REL_F32


def test_compose_random_geometries_batched():
    """Twelve seeded random geometries (groups, stride, dilation, k up to 5,
    ragged channel counts) composed in one batched call."""
    geoms = random_geometries(77, 12, aoc.param_shapes)
    print(f"[compose random] {geoms}", flush=True)
    layers, refs = [], []
    for i, geom in enumerate(geoms):
        cin, cout, k, s, d, g = geom
        rko, proj = oracle_factors(geom, 300 + i)
        kern = torch.empty(cout, cin // g, k, k, device=DEV)
        layers.append(dict(geom=geom, rko=to_dev(rko), proj=to_dev(proj) if proj is not None else None, kernel=kern))
        refs.append(aoc.aoc_kernel(rko.astype(np.float64), None if proj is None else proj.astype(np.float64), *geom))
    orth.orth_build_conv_kernels_batched(layers)
    torch.cuda.synchronize()
    for L, ref, geom in zip(layers, refs, geoms):
        assert checks.relative_difference(to_f64(L["kernel"]), ref) <= REL_F32, geom


def test_compose_batched_bf16_storage():
    layers, refs = [], []
    for i, geom in enumerate(COMPOSE_GEOMS[:5]):
        cin, cout, k, s, d, g = geom
        rko, proj = oracle_factors(geom, 50 + i)
        rko_b = torch.from_numpy(rko).to(torch.bfloat16).to(DEV)
        proj_b = torch.from_numpy(proj).to(torch.bfloat16).to(DEV) if proj is not None else None
        kern = torch.empty(cout, cin // g, k, k, dtype=torch.bfloat16, device=DEV)
        layers.append(dict(geom=geom, rko=rko_b, proj=proj_b, kernel=kern))
        refs.append(aoc.aoc_kernel(to_f64(rko_b), None if proj_b is None else to_f64(proj_b), *geom))
    orth.orth_build_conv_kernels_batched(layers)
    torch.cuda.synchronize()
    for L, ref in zip(layers, refs):
        # inputs are exact bf16 values; arithmetic fp32; one final bf16 rounding
        assert checks.relative_difference(to_f64(L["kernel"]), ref) <= 4e-3


# ----------------------------------------------------------------- checks --

def test_check_gram_parity():
    shapes = [(16, 8), (8, 16), (100, 70), (300, 200), (64, 64)]
    st = stored(108, shapes)
    mats = [to_dev(s) for s in st]
    dev = orth.orth_check_norm_gram(mats).cpu().numpy()
    for d, s in zip(dev, st):
        ref = checks.gram_deviation(s.astype(np.float64))
        assert abs(d - ref) <= 1e-5 * max(1.0, ref)


@pytest.mark.parametrize("geom,hw,adjoint", [((16, 16, 3, 1, 1, 1), 16, False), ((8, 16, 3, 2, 1, 1), 8, True),
                                             ((12, 12, 3, 1, 2, 3), 8, False), ((4, 16, 2, 2, 1, 1), 8, False)])
def test_check_conv_parity(geom, hw, adjoint):
    cin, cout, k, s, d, g = geom
    rng = np.random.default_rng(7)
    kern = rng.standard_normal((cout, cin // g, k, k)).astype(np.float32)
    if adjoint:
        x = rng.standard_normal((3, cout, hw // s, hw // s)).astype(np.float32)
        ref = checks.conv_adjoint_norm_ratios(kern.astype(np.float64), x, (hw, hw), s, d, g)
    else:
        x = rng.standard_normal((3, cin, hw, hw)).astype(np.float32)
        ref = checks.conv_norm_ratios(kern.astype(np.float64), x, s, d, g)
    got = orth.orth_check_norm_conv(to_dev(kern), geom, to_dev(x), adjoint=adjoint).cpu().numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-5)


# ------------------------------------------------------ whole workloads --

def run_workload_layers(w, iters, compute="f32"):
    """Orthogonalize all factors of a workload in one call, then build every
    conv kernel in one call.  Returns (raw stored matrices, GPU outputs,
    GPU kernels per layer)."""
    st = wl.all_matrices(w)
    outs, status = gpu_orthogonalize(st, iters, compute=compute)
    assert np.all(status == 0)
    kernels, layers = [], []
    for layer, (a, b) in zip(w.layers, wl.layer_matrix_ranges(w)):
        if not isinstance(layer, wl.ConvLayer):
            kernels.append(None)
            continue
        g, npj = layer.groups, layer.n_proj
        per = 1 + npj
        rko = torch.stack([outs[a + j * per] for j in range(g)]).contiguous()
        proj = torch.stack([torch.stack(outs[a + j * per + 1: a + (j + 1) * per]) for j in range(g)]).contiguous() \
            if npj else None
        kern = torch.empty(layer.cout, layer.c, layer.k, layer.k, device=DEV)
        layers.append(dict(geom=(layer.cin, layer.cout, layer.k, layer.stride, layer.dilation, layer.groups),
                           rko=rko, proj=proj, kernel=kern))
        kernels.append(kern)
    orth.orth_build_conv_kernels_batched(layers)
    torch.cuda.synchronize()
    return st, outs, kernels


def oracle_layer(w, layer, st, a, iters):
    g, npj = layer.groups, layer.n_proj
    per = 1 + npj
    x = oracle_inputs(st[a:a + g * per])
    raw_r = np.stack([x[j * per] for j in range(g)])
    raw_p = np.stack([np.stack(x[j * per + 1:(j + 1) * per]) for j in range(g)]) if npj else None
    return aoc.aoc_layer(raw_r, raw_p, layer.cin, layer.cout, layer.k, layer.stride, layer.dilation, layer.groups,
                         iters)


def test_workload_conv3x3_c16():
    """One 3x3 16->16 layer: kernel parity at the configured T, then at a
    converged T the Toeplitz spectrum on 8x8 inputs and norm preservation on
    an 8x16x16x16 batch."""
    w = wl.WORKLOADS["conv3x3_c16"]
    for iters in (w.iters, t_conv(oracle_inputs(wl.all_matrices(w)))):
        st, outs, kernels = run_workload_layers(w, iters)
        ref = oracle_layer(w, w.layers[0], st, 0, iters)
        got = to_f64(kernels[0])
        assert checks.relative_difference(got, ref) <= REL_F32
    sv = conv.toeplitz_singular_values(got, 8, 8)
    assert np.max(np.abs(sv - 1)) <= 1e-4
    x = wl.check_batch(w)
    ratios = orth.orth_check_norm_conv(kernels[0], (16, 16, 3, 1, 1, 1), to_dev(x)).cpu().numpy()
    assert np.max(np.abs(ratios - 1)) <= 1e-5


def test_workload_mixed_gds19():
    w = wl.WORKLOADS["mixed_gds19"]
    st_all = oracle_inputs(wl.all_matrices(w))
    for iters in (w.iters, t_conv(st_all)):
        st, outs, kernels = run_workload_layers(w, iters)
        for li, (layer, (a, b)) in enumerate(zip(w.layers, wl.layer_matrix_ranges(w))):
            if li in (0, 1, 10, 11, 15):     # one of each repeated layer kind
                ref = oracle_layer(w, layer, st, a, iters)
                assert checks.relative_difference(to_f64(kernels[li]), ref) <= REL_F32, (li, iters)
    # norm preservation on 4 x cin x 32 x 32 at the converged T
    for li in (0, 10, 15):
        layer = w.layers[li]
        x = wl.check_batch(w, (4, layer.cin, 32, 32))
        geom = (layer.cin, layer.cout, layer.k, layer.stride, layer.dilation, layer.groups)
        r = orth.orth_check_norm_conv(kernels[li], geom, to_dev(x)).cpu().numpy()
        assert np.max(np.abs(r - 1)) <= 1e-5, li


def test_workload_cifar_stack12():
    """Every layer of the CIFAR-like stack (fp32, T = 15; all 54 factors in
    one call, all 12 kernels in one call) against the oracle's whole chain
    from the raw parameters: kernels up to 256 channels in full, the
    512-wide ones on sampled output channels (K = R ⊛ B is linear in R row
    by row, App. B.1).  Then the same at T_conv: max |G - I| of all 54
    factors within the fp32 bound, and norm preservation of a circular conv
    input at every width."""
    w = wl.WORKLOADS["cifar_stack12"]
    st_all = oracle_inputs(wl.all_matrices(w))
    T_conv = t_conv(st_all)
    for iters in (w.iters, T_conv):
        print(f"[cifar] T = {iters}", flush=True)
        st, outs, kernels = run_workload_layers(w, iters)
        for li, (layer, (a, b)) in enumerate(zip(w.layers, wl.layer_matrix_ranges(w))):
            fac = [bjorck.bjorck(m, iters) for m in st_all[a:b]]
            got = to_f64(kernels[li])
            if layer.cout <= 256:
                ref = aoc.aoc_kernel(fac[0][None], np.stack(fac[1:])[None], layer.cin, layer.cout, layer.k,
                                     layer.stride, layer.dilation, layer.groups)
                rel = checks.relative_difference(got, ref)
            else:
                rows = sorted({0, 63, 64, 200, 255, 256, 383, 448, layer.cout - 1})
                ref = aoc.compose_group(fac[0][rows], fac[1:], layer.c, layer.k, layer.stride)
                rel = checks.relative_difference(got[rows], ref)
            assert rel <= REL_F32, (li, iters, rel)
        if iters == T_conv:
            for i, o in enumerate(outs):
                assert checks.gram_deviation(to_f64(o)) <= ORTH_F32, i
            for li in (0, 2, 3, 4, 8, 11):
                # stride-2 transitions (cout = 2 cin) map onto fewer output
                # values: their rows are orthonormal, so the transposed conv
                # preserves the norm (an input on the output grid)
                layer = w.layers[li]
                geom = (layer.cin, layer.cout, layer.k, layer.stride, layer.dilation, layer.groups)
                adjoint = layer.stride > 1
                shape = (2, layer.cout, 8, 8) if adjoint else (2, layer.cin, 16, 16)
                x = wl.check_batch(w, shape)
                r = orth.orth_check_norm_conv(kernels[li], geom, to_dev(x), adjoint=adjoint).cpu().numpy()
                assert np.max(np.abs(r - 1)) <= 1e-5, (li, r)


def test_diagnostic_switches():
    """ORTH_LOG=2 prints every call's plan and every launch; ORTH_DEBUG_SYNC=1
    synchronizes after each launch and reports it done.  Run in a child
    process (the switches are read once per process)."""
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    code = ("import sys, torch; sys.path.insert(0, %r); sys.path.insert(0, %r)\n"
            "from gpu_util import gpu_orthogonalize\n"
            "from test_gpu_parity import stored\n"
            "outs, status = gpu_orthogonalize(stored(5, [(300, 200), (40, 20)]), 3)\n"
            "assert (status == 0).all()\n" % (root, os.path.join(root, "tests")))
    env = dict(os.environ, ORTH_LOG="2", ORTH_DEBUG_SYNC="1")
    p = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True, timeout=300)
    assert p.returncode == 0, p.stderr[-2000:]
    err = p.stderr
    assert "[orth] orth_orthogonalize_batched: 2 matrices" in err, err[-2000:]
    assert "[orth] launch bjorck_gram_f32" in err and "[orth] ORTH_DEBUG_SYNC: bjorck_gram_f32 done" in err
    assert "failed" not in err
