"""AOC kernel construction, float64, written from Appendix B.1.

The paper builds an explicit orthogonal k x k kernel as

    AOC = RKO ⊛ K_BCOP

where ⊛ is the block-convolution (kernel-on-kernel) operator: the kernel of
the composition of two convolutions.  The paper defers the AOC details to a
companion paper, so this module fixes one reading that is provably
orthogonal:

* c = cin / groups channels per group, k' = k - s + 1 (valid iff k >= s).
* RKO factor: an s x s kernel with stride s whose (cout/g) x (c s^2)
  reshape M is the Björck output; R[o, i, a, b] = M[o, i s^2 + a s + b].
* BCOP factor (stride 1, c -> c channels): the product of k'-1 horizontal
  1x2 blocks and k'-1 vertical 2x1 blocks.  Each block is built from a
  symmetric projector P = V V^T, V the c x floor(c/2) Björck output with
  orthonormal columns: horizontal taps [0,0] = P, [0,1] = I - P; vertical
  taps [0,0] = P, [1,0] = I - P.  Such a block is unitary at every
  frequency because P is idempotent and symmetric.
* Order: K_g = R ⊛ Bh(P_1) ⊛ ... ⊛ Bh(P_{k'-1}) ⊛ Bv(Q_1) ⊛ ... ⊛ Bv(Q_{k'-1}),
  i.e. the BCOP blocks act on the input first and the strided RKO last.
* Groups: group j fills output rows [j cout/g, (j+1) cout/g) of the
  (cout, c, k, k) OIHW tensor (Appendix B.1, native grouped convolution).
* Dilation is a property of how the kernel is applied, not of its values
  (Appendix B.1, dilation paragraph); stride together with dilation is
  accepted only when gcd(s, d) = 1.

Pins: P5 (projector algebra, associativity, identity, reductions k = s),
P6 (Toeplitz SVD), P7 (FFT SVD), P8 (norm preservation) and the
composition-equals-conv-of-conv check against torch's CPU conv2d.
"""

import math

import numpy as np

from . import bjorck as _bj


class GeometryError(ValueError):
    """Raised for a geometry the construction rejects.  ``kind`` is
    "invalid" (malformed arguments) or "unsupported" (a valid request that
    cannot be made orthogonal by this construction)."""

    def __init__(self, kind, msg):
        super().__init__(msg)
        self.kind = kind


def validate_geometry(cin, cout, k, stride, dilation, groups):
    """Reject malformed and impossible configurations (Section 4: impossible
    configurations must be rejected; Appendix B.1: valid iff k >= s)."""
    vals = (cin, cout, k, stride, dilation, groups)
    if any(int(v) != v for v in vals):
        raise GeometryError("invalid", "all sizes must be integers")
    if min(vals) < 1:
        raise GeometryError("invalid", "all sizes must be >= 1")
    if cin % groups or cout % groups:
        raise GeometryError("invalid", "cin and cout must be divisible by groups")
    if k < stride:
        raise GeometryError("unsupported", "kernel size must be >= stride")
    if stride > 1 and math.gcd(stride, dilation) != 1:
        raise GeometryError("unsupported", "stride > 1 needs gcd(stride, dilation) == 1")
    c = cin // groups
    if k - stride + 1 > 1 and c < 2:
        raise GeometryError("unsupported", "BCOP blocks need at least 2 channels per group")


def param_shapes(cin, cout, k, stride, dilation, groups):
    """Shapes of the free parameters of one group: the RKO matrix and the
    projector factors.  Returns (rko_rows, rko_cols, n_proj, proj_rows, proj_cols)."""
    validate_geometry(cin, cout, k, stride, dilation, groups)
    c = cin // groups
    kp = k - stride + 1
    return cout // groups, c * stride * stride, 2 * (kp - 1), c, c // 2


def rko_kernel(m, c, stride):
    """Reshape the (cout/g) x (c s^2) matrix into the s x s RKO kernel."""
    m = np.asarray(m, dtype=np.float64)
    return m.reshape(m.shape[0], c, stride, stride).copy()


def projector(v):
    """P = V V^T for V with orthonormal columns."""
    v = np.asarray(v, dtype=np.float64)
    return v @ v.T


def block_h(p):
    """Horizontal 1x2 BCOP block of a c x c projector."""
    c = p.shape[0]
    blk = np.zeros((c, c, 1, 2))
    blk[:, :, 0, 0] = p
    blk[:, :, 0, 1] = np.eye(c) - p
    return blk


def block_v(p):
    """Vertical 2x1 BCOP block of a c x c projector."""
    c = p.shape[0]
    blk = np.zeros((c, c, 2, 1))
    blk[:, :, 0, 0] = p
    blk[:, :, 1, 0] = np.eye(c) - p
    return blk


def block_conv(a, b):
    """Block-convolution operator: the kernel of conv(A, conv(B, .)).

    For cross-correlation kernels A (o, m, ha, wa) and B (m, i, hb, wb):
        (A ⊛ B)[o, i, y, x] = sum_m sum_{p,q} A[o, m, p, q] B[m, i, y-p, x-q]
    with output size (ha+hb-1, wa+wb-1).  Plain loops over taps.
    """
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    if a.shape[1] != b.shape[0]:
        raise ValueError("inner channel counts differ")
    ha, wa = a.shape[2:]
    hb, wb = b.shape[2:]
    out = np.zeros((a.shape[0], b.shape[1], ha + hb - 1, wa + wb - 1))
    for p in range(ha):
        for q in range(wa):
            for r in range(hb):
                for t in range(wb):
                    out[:, :, p + r, q + t] += a[:, :, p, q] @ b[:, :, r, t]
    return out


def identity_kernel(c):
    """The neutral element of ⊛: a 1x1 identity kernel."""
    return np.eye(c).reshape(c, c, 1, 1)


def compose_group(rko_mat, proj_mats, c, k, stride):
    """Explicit kernel of one group from already-orthogonalized factors.

    ``rko_mat``: (cout/g) x (c s^2); ``proj_mats``: 2(k'-1) matrices of
    shape c x floor(c/2), horizontal blocks first, then vertical blocks.
    """
    kp = k - stride + 1
    if len(proj_mats) != 2 * (kp - 1):
        raise ValueError("expected %d projector factors" % (2 * (kp - 1)))
    kern = rko_kernel(rko_mat, c, stride)
    for j in range(kp - 1):
        kern = block_conv(kern, block_h(projector(proj_mats[j])))
    for j in range(kp - 1):
        kern = block_conv(kern, block_v(projector(proj_mats[kp - 1 + j])))
    return kern


def aoc_kernel(rko, proj, cin, cout, k, stride, dilation, groups):
    """Compose the (cout, cin/g, k, k) kernel from orthogonalized factors.

    ``rko``: (g, cout/g, c s^2); ``proj``: (g, 2(k'-1), c, floor(c/2))
    (may be None or empty when k == s).
    """
    rr, rc, nproj, pr, pc = param_shapes(cin, cout, k, stride, dilation, groups)
    rko = np.asarray(rko, dtype=np.float64).reshape(groups, rr, rc)
    if nproj:
        proj = np.asarray(proj, dtype=np.float64).reshape(groups, nproj, pr, pc)
    c = cin // groups
    out = np.zeros((cout, c, k, k))
    for j in range(groups):
        pm = [proj[j, t] for t in range(nproj)] if nproj else []
        out[j * rr:(j + 1) * rr] = compose_group(rko[j], pm, c, k, stride)
    return out


def aoc_layer(raw_rko, raw_proj, cin, cout, k, stride, dilation, groups, iters, beta=0.5):
    """Full parametrization of one layer from raw parameters: Frobenius
    pre-scaling and Björck on every factor, then the composition."""
    rr, rc, nproj, pr, pc = param_shapes(cin, cout, k, stride, dilation, groups)
    raw_rko = np.asarray(raw_rko, dtype=np.float64).reshape(groups, rr, rc)
    rko = np.stack([_bj.bjorck(raw_rko[j], iters, beta) for j in range(groups)])
    proj = None
    if nproj:
        raw_proj = np.asarray(raw_proj, dtype=np.float64).reshape(groups, nproj, pr, pc)
        proj = np.stack([np.stack([_bj.bjorck(raw_proj[j, t], iters, beta)
                                   for t in range(nproj)]) for j in range(groups)])
    return aoc_kernel(rko, proj, cin, cout, k, stride, dilation, groups)
