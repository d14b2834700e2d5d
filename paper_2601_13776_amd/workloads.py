"""Seeded synthetic workloads shaped like the paper's backbones.

This module only describes layer stacks and draws their free parameters; it
contains none of the method's arithmetic.  Both the HIP path (tests, bench)
and the CPU oracle receive their inputs from here.

Every matrix is drawn independently from ``numpy.random.default_rng`` seeded
with ``[workload_seed, matrix_index]`` so any single matrix can be
regenerated on its own (the CPU baseline samples a few matrices of the large
workloads).  Entries are N(0, 1/fan_in) with fan_in = number of stored
columns, drawn in float64, then rounded to float32 or to bfloat16
(round-to-nearest-even).  The scale is immaterial after Frobenius
pre-scaling; only the seed and the shape matter.

Matrix order inside a workload: layer, then group, then the RKO matrix, then
the horizontal projector factors, then the vertical ones.
"""

from dataclasses import dataclass, field
import hashlib
import math

import numpy as np


@dataclass(frozen=True)
class ConvLayer:
    cin: int
    cout: int
    k: int
    stride: int = 1
    dilation: int = 1
    groups: int = 1

    @property
    def c(self):
        return self.cin // self.groups

    @property
    def n_proj(self):
        return 2 * (self.k - self.stride)

    def matrix_shapes(self):
        """(rows, cols) of every free matrix of this layer, in draw order."""
        out = []
        for _ in range(self.groups):
            out.append((self.cout // self.groups, self.c * self.stride * self.stride))
            out.extend([(self.c, self.c // 2)] * self.n_proj)
        return out


@dataclass(frozen=True)
class DenseLayer:
    rows: int
    cols: int

    def matrix_shapes(self):
        return [(self.rows, self.cols)]


@dataclass(frozen=True)
class Workload:
    name: str
    seed: int
    dtype: str            # "f32" or "bf16": storage of the raw parameters
    iters: int
    layers: tuple
    stress_row_fraction: float = 0.0
    stress_scale: float = 1.0
    check_input: tuple = field(default=())     # (N, C, H, W) of a norm-check batch

    def matrix_shapes(self):
        out = []
        for layer in self.layers:
            out.extend(layer.matrix_shapes())
        return out

    @property
    def n_layers(self):
        return len(self.layers)


def _cifar_stack():
    widths = [64, 64, 128, 128, 256, 256, 256, 256, 512, 512, 512, 512]
    layers = []
    prev = widths[0]
    for w in widths:
        layers.append(ConvLayer(prev, w, 3, stride=2 if w != prev else 1))
        prev = w
    return tuple(layers)


def _mixed_stack():
    layers = [ConvLayer(256, 256, 3, groups=4)] * 10
    layers += [ConvLayer(256, 256, 3, dilation=2)] * 5
    layers += [ConvLayer(128, 512, 2, stride=2)] * 4
    return tuple(layers)


def _imagenet_stack():
    layers = []
    for c in (128, 256, 512, 1024):
        layers += [ConvLayer(c, c, 3)] * 4
    layers += [DenseLayer(1024, 1024)] * 4
    layers += [DenseLayer(2048, 2048)] * 4
    layers.append(DenseLayer(1000, 2048))
    return tuple(layers)


def _stress_batch():
    return tuple([DenseLayer(4096, 4096)] * 64 + [DenseLayer(32, 32)] * 4096)


WORKLOADS = {
    # one 3x3 16->16 orthogonal conv, fp32, 12 iterations
    "conv3x3_c16": Workload("conv3x3_c16", 1, "f32", 12, (ConvLayer(16, 16, 3),),
                            check_input=(8, 16, 16, 16)),
    # CIFAR-like stack of 12 3x3 layers (64..512), stride 2 at width changes
    "cifar_stack12": Workload("cifar_stack12", 2, "f32", 15, _cifar_stack()),
    # grouped / dilated / strided mix
    "mixed_gds19": Workload("mixed_gds19", 3, "f32", 15, _mixed_stack(),
                            check_input=(4, 256, 32, 32)),
    # ImageNet-like backbone parametrization, bf16 operands
    "imagenet_backbone25": Workload("imagenet_backbone25", 4, "bf16", 20, _imagenet_stack()),
    # stress batch: 64 x 4096^2 + 4096 x 32^2, 5% of rows scaled by 100
    "stress_4096x64_32x4096": Workload("stress_4096x64_32x4096", 5, "bf16", 25, _stress_batch(),
                                       stress_row_fraction=0.05, stress_scale=100.0),
}

WORKLOAD_ORDER = ["conv3x3_c16", "cifar_stack12", "mixed_gds19",
                  "imagenet_backbone25", "stress_4096x64_32x4096"]


def f32_to_bf16_bits(a):
    """Round float32 values to bfloat16 (nearest, ties to even); returns the
    raw uint16 bit patterns (the layout of torch.bfloat16)."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    nan = np.isnan(a)
    out = rounded.astype(np.uint16)
    out[nan] = 0x7FC0
    return out


def bf16_bits_to_f64(bits):
    """Exact widening of bfloat16 bit patterns."""
    b = np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def draw_matrix(workload, index, rows, cols):
    """Draw matrix ``index`` of ``workload`` in float64 (before rounding)."""
    rng = np.random.default_rng([workload.seed, index])
    m = rng.standard_normal((rows, cols)) / math.sqrt(cols)
    if workload.stress_row_fraction > 0.0:
        n_rows = int(round(workload.stress_row_fraction * rows))
        if n_rows:
            picked = rng.choice(rows, size=n_rows, replace=False)
            m[picked] *= workload.stress_scale
    return m


def stored_matrix(workload, index, rows, cols):
    """The matrix as handed to the library: float32 array, or uint16 bf16
    bit patterns when the workload is bf16."""
    m = draw_matrix(workload, index, rows, cols)
    if workload.dtype == "bf16":
        return f32_to_bf16_bits(m.astype(np.float32))
    return m.astype(np.float32)


def as_f64(stored):
    """The exact float64 value of a stored matrix (what the oracle sees)."""
    if stored.dtype == np.uint16:
        return bf16_bits_to_f64(stored)
    return stored.astype(np.float64)


def all_matrices(workload, indices=None):
    """List of stored matrices (optionally only the given indices)."""
    shapes = workload.matrix_shapes()
    idx = range(len(shapes)) if indices is None else indices
    return [stored_matrix(workload, i, *shapes[i]) for i in idx]


def layer_matrix_ranges(workload):
    """For every layer, the [start, end) range of its matrices in draw order."""
    out, pos = [], 0
    for layer in workload.layers:
        n = len(layer.matrix_shapes())
        out.append((pos, pos + n))
        pos += n
    return out


def check_batch(workload, shape=None, seed_offset=100):
    """N(0,1) float32 input for a norm check, seeded with seed + 100."""
    shape = shape or workload.check_input
    rng = np.random.default_rng(workload.seed + seed_offset)
    return rng.standard_normal(shape).astype(np.float32)


def sha256_of(arrays):
    h = hashlib.sha256()
    for a in arrays:
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def algorithmic_bjorck_flops(shapes, iters):
    """sum over matrices of 4 m n min(m, n) T: two dense products per step."""
    return sum(4 * r * c * min(r, c) * iters for r, c in shapes)
