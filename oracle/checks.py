"""Gate quantities computed on the CPU in float64 (Section 4: orthogonality
checks; Appendix C: norm and singular-value tolerances)."""

import numpy as np

from . import conv as _conv


def gram_deviation(w):
    """max |G - I| with G the smaller Gram matrix (W^T W for rows >= cols,
    W W^T otherwise)."""
    w = np.asarray(w, dtype=np.float64)
    rows, cols = w.shape
    g = w.T @ w if rows >= cols else w @ w.T
    return float(np.max(np.abs(g - np.eye(g.shape[0]))))


def relative_difference(a, b):
    """||a - b||_F / ||b||_F in float64."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = np.sqrt(np.sum(b * b))
    return float(np.sqrt(np.sum((a - b) ** 2)) / den) if den else float(np.sqrt(np.sum(a * a)))


def conv_norm_ratios(kernel, x, stride=1, dilation=1, groups=1):
    """||conv_circ(K, x_n)|| / ||x_n|| for every sample of the batch."""
    y = _conv.conv_circular(kernel, x, stride, dilation, groups)
    n = x.shape[0]
    num = np.sqrt(np.sum(np.asarray(y).reshape(n, -1) ** 2, axis=1))
    den = np.sqrt(np.sum(np.asarray(x, dtype=np.float64).reshape(n, -1) ** 2, axis=1))
    return num / den


def conv_adjoint_norm_ratios(kernel, y, in_hw, stride=1, dilation=1, groups=1):
    """||conv_circ^T(K, y_n)|| / ||y_n|| for every sample."""
    x = _conv.conv_circular_adjoint(kernel, y, in_hw, stride, dilation, groups)
    n = y.shape[0]
    num = np.sqrt(np.sum(x.reshape(n, -1) ** 2, axis=1))
    den = np.sqrt(np.sum(np.asarray(y, dtype=np.float64).reshape(n, -1) ** 2, axis=1))
    return num / den


def tile_relative_differences(a, b, tile=256):
    """||a_T - b_T||_F / ||b_T||_F for every tile x tile block T of the
    matrices (ragged blocks at the right and bottom edges included; a block
    whose reference is all zero reports ||a_T||_F).  Returned as a
    (row blocks, column blocks) array, so that an error confined to a few
    blocks stands out against the whole-matrix relative difference."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    if a.shape != b.shape:
        raise ValueError("shapes differ")
    rows, cols = b.shape
    nr, nc = -(-rows // tile), -(-cols // tile)
    out = np.zeros((nr, nc))
    for i in range(nr):
        for j in range(nc):
            out[i, j] = relative_difference(a[i * tile:(i + 1) * tile, j * tile:(j + 1) * tile],
                                            b[i * tile:(i + 1) * tile, j * tile:(j + 1) * tile])
    return out
