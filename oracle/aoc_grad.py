"""Vector-Jacobian product of the AOC kernel construction, float64.

The forward construction (Appendix B.1, AOC = RKO ⊛ K_BCOP with the BCOP
factor a chain of 1x2 and 2x1 projector blocks) is bilinear in each ⊛ step:

    <dC, A ⊛ B> = sum_{p,q,r,t} <dC[:, :, p+r, q+t], A[:, :, p, q] B[:, :, r, t]>,

so for C = A ⊛ B

    dA[:, :, p, q] = sum_{r,t} dC[:, :, p+r, q+t] B[:, :, r, t]^T,
    dB[:, :, r, t] = sum_{p,q} A[:, :, p, q]^T dC[:, :, p+r, q+t].

A horizontal block has taps P and I - P, so dP = dB[0,0] - dB[0,1] (vertical:
dB[0,0] - dB[1,0]); P = V V^T gives dV = (dP + dP^T) V; the RKO reshape is
undone by a reshape.  The chain is walked backwards over recomputed
intermediates, plain loops over taps.

Pins (tests/test_oracle_grad_pins.py): the adjoint identity of the part
linear in the RKO factor, central finite differences in the projector
factors and through the whole layer (Björck included), and per-factor scale
invariance of the raw-parameter gradient.
"""

import numpy as np

from . import aoc as _aoc
from . import bjorck as _bj
from . import bjorck_grad as _bg


def block_conv_vjp(a, b, dc):
    """(dL/dA, dL/dB) for C = A ⊛ B given dL/dC."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    dc = np.asarray(dc, dtype=np.float64)
    ha, wa = a.shape[2:]
    hb, wb = b.shape[2:]
    da = np.zeros(a.shape)
    db = np.zeros(b.shape)
    for p in range(ha):
        for q in range(wa):
            for r in range(hb):
                for t in range(wb):
                    g = dc[:, :, p + r, q + t]
                    da[:, :, p, q] += g @ b[:, :, r, t].T
                    db[:, :, r, t] += a[:, :, p, q].T @ g
    return da, db


def block_h_vjp(db):
    """dL/dP of the horizontal block (taps P, I - P)."""
    return db[:, :, 0, 0] - db[:, :, 0, 1]


def block_v_vjp(db):
    """dL/dP of the vertical block (taps P, I - P)."""
    return db[:, :, 0, 0] - db[:, :, 1, 0]


def projector_vjp(v, dp):
    """dL/dV of P = V V^T."""
    v = np.asarray(v, dtype=np.float64)
    return (dp + dp.T) @ v


def compose_group_vjp(rko_mat, proj_mats, c, k, stride, dk):
    """Gradient of one group's composed kernel with respect to its
    orthogonalized factors: returns (d rko_mat, [d proj_mat ...])."""
    kp = k - stride + 1
    if len(proj_mats) != 2 * (kp - 1):
        raise ValueError("expected %d projector factors" % (2 * (kp - 1)))
    blocks = []
    for j in range(kp - 1):
        blocks.append(_aoc.block_h(_aoc.projector(proj_mats[j])))
    for j in range(kp - 1):
        blocks.append(_aoc.block_v(_aoc.projector(proj_mats[kp - 1 + j])))
    chain = [_aoc.rko_kernel(rko_mat, c, stride)]
    for blk in blocks:
        chain.append(_aoc.block_conv(chain[-1], blk))
    g = np.asarray(dk, dtype=np.float64)
    dproj = [None] * len(blocks)
    for j in range(len(blocks) - 1, -1, -1):
        g, dblk = block_conv_vjp(chain[j], blocks[j], g)
        dp = block_h_vjp(dblk) if j < kp - 1 else block_v_vjp(dblk)
        dproj[j] = projector_vjp(proj_mats[j], dp)
    return g.reshape(g.shape[0], -1), dproj


def aoc_kernel_vjp(rko, proj, cin, cout, k, stride, dilation, groups, dk):
    """Gradient of aoc_kernel with respect to its factors.

    Returns (d_rko of shape (g, cout/g, c s^2), d_proj of shape
    (g, 2(k'-1), c, floor(c/2)) or None when k == s)."""
    rr, rc, nproj, pr, pc = _aoc.param_shapes(cin, cout, k, stride, dilation, groups)
    c = cin // groups
    rko = np.asarray(rko, dtype=np.float64).reshape(groups, rr, rc)
    dk = np.asarray(dk, dtype=np.float64).reshape(cout, c, k, k)
    if nproj:
        proj = np.asarray(proj, dtype=np.float64).reshape(groups, nproj, pr, pc)
    drko = np.zeros((groups, rr, rc))
    dproj = np.zeros((groups, nproj, pr, pc)) if nproj else None
    for j in range(groups):
        pm = [proj[j, t] for t in range(nproj)] if nproj else []
        dr, dps = compose_group_vjp(rko[j], pm, c, k, stride, dk[j * rr:(j + 1) * rr])
        drko[j] = dr
        for t in range(nproj):
            dproj[j, t] = dps[t]
    return drko, dproj


def aoc_layer_vjp(raw_rko, raw_proj, cin, cout, k, stride, dilation, groups, iters, dk, beta=0.5):
    """Gradient of aoc_layer (Frobenius pre-scaling, Björck on every factor,
    composition) with respect to the raw parameters."""
    rr, rc, nproj, pr, pc = _aoc.param_shapes(cin, cout, k, stride, dilation, groups)
    raw_rko = np.asarray(raw_rko, dtype=np.float64).reshape(groups, rr, rc)
    rko = np.stack([_bj.bjorck(raw_rko[j], iters, beta) for j in range(groups)])
    proj = None
    if nproj:
        raw_proj = np.asarray(raw_proj, dtype=np.float64).reshape(groups, nproj, pr, pc)
        proj = np.stack([np.stack([_bj.bjorck(raw_proj[j, t], iters, beta)
                                   for t in range(nproj)]) for j in range(groups)])
    drko, dproj = aoc_kernel_vjp(rko, proj, cin, cout, k, stride, dilation, groups, dk)
    g_rko = np.stack([_bg.bjorck_vjp(raw_rko[j], drko[j], iters, beta) for j in range(groups)])
    g_proj = None
    if nproj:
        g_proj = np.stack([np.stack([_bg.bjorck_vjp(raw_proj[j, t], dproj[j, t], iters, beta)
                                     for t in range(nproj)]) for j in range(groups)])
    return g_rko, g_proj
