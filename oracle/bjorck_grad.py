"""Vector-Jacobian product of the Björck parametrization, float64.

For the Appendix A.5 step W' = (1 + beta) W - beta W W^T W and an upstream
gradient Y = dL/dW', differentiating <Y, W'> gives, for rows >= cols with
G = W^T W,

    dL/dW = Y ((1 + beta) I - beta G) - beta W (W^T Y + Y^T W),

and for rows < cols with H = W W^T,

    dL/dW = ((1 + beta) I - beta H) Y - beta (Y W^T + W Y^T) W.

The Frobenius pre-scaling W_0 = W / s, s = ||W||_F, contributes
dL/dW = (Y_0 - <Y_0, W_0> W_0) / s.  The steps are chained from the last
iterate back to the input; the forward iterates are recomputed here.

Pins (tests/test_oracle_grad_pins.py): central finite differences, and
torch.autograd through an independent float64 forward.
"""

import numpy as np

from . import bjorck as _bj


def bjorck_step_vjp(w, y, beta=0.5):
    """dL/dW of one Björck step at iterate W given dL/dW' = Y."""
    w = np.asarray(w, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    rows, cols = w.shape
    if rows >= cols:
        g = w.T @ w
        return (1.0 + beta) * y - beta * (y @ g) - beta * (w @ (w.T @ y + y.T @ w))
    h = w @ w.T
    return (1.0 + beta) * y - beta * (h @ y) - beta * ((y @ w.T + w @ y.T) @ w)


def bjorck_vjp(w, grad_out, iters, beta=0.5, prescale="frobenius"):
    """dL/dW for L depending on W through bjorck(W, iters, beta, prescale),
    given dL/dW_T = grad_out.  Zero input: zero gradient; non-finite input:
    all-NaN gradient (mirroring the forward's statuses)."""
    w = np.asarray(w, dtype=np.float64)
    y = np.asarray(grad_out, dtype=np.float64)
    if prescale == "frobenius":
        w0, status = _bj.frobenius_prescale(w)
        if status == _bj.STATUS_NONFINITE:
            return np.full(w.shape, np.nan)
        if status == _bj.STATUS_ZERO:
            return np.zeros(w.shape)
        s = np.sqrt(np.sum(w * w))
    elif prescale == "none":
        if not np.all(np.isfinite(w)):
            return np.full(w.shape, np.nan)
        w0, s = w, None
    else:
        raise ValueError("prescale must be 'frobenius' or 'none'")
    iterates = [w0]
    for _ in range(iters):
        iterates.append(_bj.bjorck_step(iterates[-1], beta))
    for t in range(iters - 1, -1, -1):
        y = bjorck_step_vjp(iterates[t], y, beta)
    if s is None:
        return y
    return (y - np.sum(y * w0) * w0) / s
