"""Circular convolution and its exact spectrum, float64.

Section 4 and Appendix C test orthogonal convolutions by (i) the explicit
SVD of the convolution's Toeplitz matrix built from impulse responses on
small (8 x 8) inputs, and (ii) scalable spectral methods; for stride 1 and
circular padding the spectrum is the union over spatial frequencies of the
singular values of the Fourier-transformed kernel (the method the paper cites
as Sedghi et al.).  Circular padding is used throughout, as in the paper's
tests.

Convention (cross-correlation, as torch.nn.functional.conv2d):

    y[n, o, u, v] = sum_{i, a, b} K[o, i, a, b]
                    x[n, g(o) c + i, (s u + d a - pl) mod H, (s v + d b - pl) mod W]

with c = cin/groups, g(o) = o // (cout/groups), total padding
P = d (k - 1) + 1 - s, pl = floor(P / 2), and output size (H/s, W/s).
This is exactly F.pad(x, (pl, P-pl, pl, P-pl), mode="circular") followed by
conv2d(stride=s, dilation=d, groups=g); the pin test checks that.
"""

import numpy as np


def _pad_left(k, stride, dilation):
    total = dilation * (k - 1) + 1 - stride
    return total // 2


def _check_sizes(kernel, x_channels, h, w, stride, dilation, groups):
    cout, c, kh, kw = kernel.shape
    if kh != kw:
        raise ValueError("square kernels only")
    if c * groups != x_channels:
        raise ValueError("input channels do not match kernel and groups")
    if h % stride or w % stride:
        raise ValueError("spatial size must be divisible by the stride")


def conv_circular(kernel, x, stride=1, dilation=1, groups=1):
    """Apply the kernel to a batch x (N, cin, H, W) with circular padding."""
    kernel = np.asarray(kernel, dtype=np.float64)
    x = np.asarray(x, dtype=np.float64)
    n, cin, h, w = x.shape
    _check_sizes(kernel, cin, h, w, stride, dilation, groups)
    cout, c, k, _ = kernel.shape
    og = cout // groups
    pl = _pad_left(k, stride, dilation)
    ho, wo = h // stride, w // stride
    rows = np.arange(ho) * stride
    cols = np.arange(wo) * stride
    y = np.zeros((n, cout, ho, wo))
    for g in range(groups):
        xg = x[:, g * c:(g + 1) * c]
        kg = kernel[g * og:(g + 1) * og]
        for a in range(k):
            ri = (rows + dilation * a - pl) % h
            for b in range(k):
                ci = (cols + dilation * b - pl) % w
                patch = xg[:, :, ri][:, :, :, ci]          # (n, c, ho, wo)
                y[:, g * og:(g + 1) * og] += np.einsum("oi,nihw->nohw", kg[:, :, a, b], patch)
    return y


def conv_circular_adjoint(kernel, y, in_hw, stride=1, dilation=1, groups=1):
    """Adjoint (transpose) of ``conv_circular`` applied to y (N, cout, H/s, W/s);
    returns (N, cin, H, W) where (H, W) = in_hw."""
    kernel = np.asarray(kernel, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    h, w = in_hw
    cout, c, k, _ = kernel.shape
    og = cout // groups
    n = y.shape[0]
    pl = _pad_left(k, stride, dilation)
    ho, wo = h // stride, w // stride
    if y.shape[1:] != (cout, ho, wo):
        raise ValueError("y has the wrong shape")
    rows = np.arange(ho) * stride
    cols = np.arange(wo) * stride
    x = np.zeros((n, c * groups, h, w))
    for g in range(groups):
        yg = y[:, g * og:(g + 1) * og]
        kg = kernel[g * og:(g + 1) * og]
        for a in range(k):
            ri = (rows + dilation * a - pl) % h
            for b in range(k):
                ci = (cols + dilation * b - pl) % w
                contrib = np.einsum("oi,nohw->nihw", kg[:, :, a, b], yg)
                for iu, r in enumerate(ri):
                    # rows of one output line map to distinct input columns
                    np.add.at(x[:, g * c:(g + 1) * c, r], (slice(None), slice(None), ci),
                              contrib[:, :, iu, :])
    return x


def toeplitz_matrix(kernel, h, w, stride=1, dilation=1, groups=1):
    """Dense matrix of the circular convolution on (cin, H, W) inputs, built
    column by column from impulse responses (Appendix C)."""
    cout, c, k, _ = kernel.shape
    cin = c * groups
    dim = cin * h * w
    basis = np.eye(dim).reshape(dim, cin, h, w)
    cols = conv_circular(kernel, basis, stride, dilation, groups)
    return cols.reshape(dim, -1).T


def toeplitz_singular_values(kernel, h, w, stride=1, dilation=1, groups=1):
    """All singular values of the convolution, sorted descending."""
    t = toeplitz_matrix(kernel, h, w, stride, dilation, groups)
    return np.linalg.svd(t, compute_uv=False)


def fft_singular_values(kernel, h, w, dilation=1, groups=1):
    """Stride-1 circular convolution spectrum: for every frequency (fu, fv),
    the singular values of sum_{a,b} K[:, :, a, b] exp(2 pi i d (a fu / H + b fv / W)),
    per group.  Sorted descending."""
    kernel = np.asarray(kernel, dtype=np.float64)
    cout, c, k, _ = kernel.shape
    og = cout // groups
    fu = np.arange(h)[:, None, None]
    fv = np.arange(w)[None, :, None]
    taps = np.arange(k)
    ph_a = np.exp(2j * np.pi * dilation * taps[None, None, :] * fu / h)   # (h,1,k)
    ph_b = np.exp(2j * np.pi * dilation * taps[None, None, :] * fv / w)   # (1,w,k)
    out = []
    for g in range(groups):
        kg = kernel[g * og:(g + 1) * og]
        # (h, w, og, c) transfer matrices
        tf = np.einsum("oiab,uxa,uxb->uxoi", kg,
                       np.broadcast_to(ph_a, (h, w, k)), np.broadcast_to(ph_b, (h, w, k)))
        out.append(np.linalg.svd(tf, compute_uv=False).ravel())
    return np.sort(np.concatenate(out))[::-1]
