"""GPU parity of the explicit-kernel convolution and its transpose
(orth_conv_apply) against the float64 oracle (oracle/conv.py), and the
orthogonality properties of transposed AOC convolutions.

Tolerance: relative Frobenius difference 1e-5 (fp32 products and sums over
c k^2 <= 4608 terms: rounding ~1e-6)."""

import numpy as np
import pytest
import torch

from oracle import aoc, bjorck, checks, conv
from paper_2601_13776_amd import orth

from gpu_util import DEV, random_geometries, to_f64

pytestmark = pytest.mark.gpu

REL = 1e-5

GEOMS = [  # (cin, cout, k, s, d, g), H
    ((16, 16, 3, 1, 1, 1), 16), ((64, 128, 3, 2, 1, 1), 16), ((32, 32, 3, 1, 1, 4), 12),
    ((32, 32, 3, 1, 2, 1), 10), ((6, 6, 5, 2, 3, 3), 12), ((24, 16, 4, 2, 1, 2), 8),
    ((4, 6, 3, 1, 1, 1), 7), ((128, 512, 2, 2, 1, 1), 8), ((100, 70, 3, 1, 1, 1), 9),
    # dilated span beyond one period of a 4 x 4 grid: the general modulo path
    ((4, 4, 5, 1, 3, 1), 4), ((8, 8, 3, 2, 5, 2), 4),
    # 128 x 128 tiles with ragged rows both ways (200 and 130 output rows)
    ((130, 200, 3, 1, 1, 1), 6),
    # a 3-channel stem and head, k = 7 (no halo path), even k with stride
    ((3, 64, 3, 1, 1, 1), 16), ((64, 3, 3, 1, 1, 1), 16), ((16, 16, 7, 1, 1, 1), 11), ((32, 64, 4, 2, 1, 1), 12),
]


def rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape).astype(np.float32)


@pytest.mark.parametrize("geom,hw", GEOMS)
def test_forward_and_transposed_parity(geom, hw):
    cin, cout, k, s, d, g = geom
    print(f"[conv apply] {geom} hw={hw}", flush=True)
    kern = rand((cout, cin // g, k, k), 1)
    x = rand((3, cin, hw, hw), 2)
    kt = torch.from_numpy(kern).to(DEV)
    y = orth.orth_conv_apply(kt, geom, torch.from_numpy(x).to(DEV))
    ref = conv.conv_circular(kern.astype(np.float64), x.astype(np.float64), s, d, g)
    assert checks.relative_difference(to_f64(y), ref) <= REL
    yy = rand((3, cout, hw // s, hw // s), 3)
    z = orth.orth_conv_apply(kt, geom, torch.from_numpy(yy).to(DEV), transposed=True)
    ref_t = conv.conv_circular_adjoint(kern.astype(np.float64), yy.astype(np.float64), (hw, hw), s, d, g)
    assert checks.relative_difference(to_f64(z), ref_t) <= REL


@pytest.mark.parametrize("case", range(10))
def test_random_geometries_parity(case):
    """Seeded random geometries (groups, stride, dilation, k up to 5, ragged
    channel counts) on random grid sizes from one stride period up, batch 2."""
    geom = random_geometries(79, 10, aoc.param_shapes)[case]
    cin, cout, k, s, d, g = geom
    hw = s * int(np.random.default_rng(case).integers(1, 8))
    print(f"[conv apply random] {geom} hw={hw}", flush=True)
    kern = rand((cout, cin // g, k, k), 10 + case)
    x = rand((2, cin, hw, hw), 20 + case)
    kt = torch.from_numpy(kern).to(DEV)
    y = orth.orth_conv_apply(kt, geom, torch.from_numpy(x).to(DEV))
    assert checks.relative_difference(to_f64(y), conv.conv_circular(kern.astype(np.float64), x.astype(np.float64),
                                                                    s, d, g)) <= REL
    yy = rand((2, cout, hw // s, hw // s), 30 + case)
    z = orth.orth_conv_apply(kt, geom, torch.from_numpy(yy).to(DEV), transposed=True)
    ref_t = conv.conv_circular_adjoint(kern.astype(np.float64), yy.astype(np.float64), (hw, hw), s, d, g)
    assert checks.relative_difference(to_f64(z), ref_t) <= REL


def test_bf16_kernel_storage():
    geom = (32, 64, 3, 2, 1, 2)
    kern = torch.from_numpy(rand((64, 16, 3, 3), 4)).to(torch.bfloat16)
    x = rand((2, 32, 12, 12), 5)
    k64 = kern.float().numpy().astype(np.float64)
    y = orth.orth_conv_apply(kern.to(DEV), geom, torch.from_numpy(x).to(DEV))
    assert checks.relative_difference(to_f64(y), conv.conv_circular(k64, x.astype(np.float64), 2, 1, 2)) <= REL
    yy = rand((2, 64, 6, 6), 6)
    z = orth.orth_conv_apply(kern.to(DEV), geom, torch.from_numpy(yy).to(DEV), transposed=True)
    ref = conv.conv_circular_adjoint(k64, yy.astype(np.float64), (12, 12), 2, 1, 2)
    assert checks.relative_difference(to_f64(z), ref) <= REL


def aoc_kernel_gpu(geom, seed):
    """Explicit AOC kernel from converged factors, composed on the GPU."""
    rr, rc, npj, pr, pc = aoc.param_shapes(*geom)
    g = geom[5]
    rng = np.random.default_rng(seed)
    rko = np.stack([bjorck.bjorck(rng.standard_normal((rr, rc)), 60) for _ in range(g)]).astype(np.float32)
    proj = None
    if npj:
        proj = np.stack([np.stack([bjorck.bjorck(rng.standard_normal((pr, pc)), 60) for _ in range(npj)])
                         for _ in range(g)]).astype(np.float32)
    cin, cout, k = geom[:3]
    kern = torch.empty(cout, cin // g, k, k, device=DEV)
    orth.orth_build_conv_kernel(torch.from_numpy(rko).to(DEV), torch.from_numpy(proj).to(DEV) if npj else None,
                                *geom, kern)
    return kern


@pytest.mark.parametrize("geom,hw", [((16, 16, 3, 1, 1, 1), 16), ((64, 128, 3, 2, 1, 1), 16),
                                     ((32, 32, 3, 1, 1, 4), 12), ((24, 48, 4, 2, 1, 2), 8),
                                     ((64, 3, 3, 1, 1, 1), 16), ((16, 16, 7, 1, 1, 1), 11)])
def test_transposed_aoc_is_isometry(geom, hw):
    """cout/g <= c s^2: the AOC conv has orthonormal rows, so its transpose
    (learnable upsampling) preserves norms and the forward conv undoes it."""
    cin, cout, k, s, d, g = geom
    assert cout // g <= (cin // g) * s * s
    kern = aoc_kernel_gpu(geom, 7)
    yy = torch.from_numpy(rand((4, cout, hw // s, hw // s), 8)).to(DEV)
    z = orth.orth_conv_apply(kern, geom, yy, transposed=True)
    back = orth.orth_conv_apply(kern, geom, z)
    torch.cuda.synchronize()
    nz = torch.linalg.vector_norm(z.flatten(1), dim=1)
    ny = torch.linalg.vector_norm(yy.flatten(1), dim=1)
    assert float(torch.max(torch.abs(nz / ny - 1))) <= REL
    assert checks.relative_difference(to_f64(back), to_f64(yy)) <= REL
    # the library's own adjoint-norm check agrees
    ratio = orth.orth_check_norm_conv(kern, geom, yy, adjoint=True)
    assert float(torch.max(torch.abs(ratio - 1))) <= REL


def test_apply_ragged_batch_and_one_pixel():
    """A single image of 1 x 1 (k = s = 1) and a batch whose pixel count is
    not a multiple of the 64-pixel tile."""
    geom = (8, 8, 1, 1, 1, 1)
    kern = rand((8, 8, 1, 1), 9)
    x = rand((1, 8, 1, 1), 10)
    y = orth.orth_conv_apply(torch.from_numpy(kern).to(DEV), geom, torch.from_numpy(x).to(DEV))
    assert checks.relative_difference(to_f64(y), conv.conv_circular(kern.astype(np.float64),
                                                                   x.astype(np.float64))) <= REL
    geom = (5, 7, 3, 1, 1, 1)
    kern = rand((7, 5, 3, 3), 11)
    x = rand((3, 5, 5, 7), 12)
    y = orth.orth_conv_apply(torch.from_numpy(kern).to(DEV), geom, torch.from_numpy(x).to(DEV))
    assert checks.relative_difference(to_f64(y), conv.conv_circular(kern.astype(np.float64),
                                                                   x.astype(np.float64))) <= REL
