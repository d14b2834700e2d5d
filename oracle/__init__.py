"""Plain, slow, float64 CPU oracle for the orthogonal-parametrization path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports this package:
only the test suite, the smoke check of ``__graft_entry__`` and the CPU
baseline leg of ``bench.py`` may call it.  It shares no code, constants or
helpers with the HIP library; both sides receive the same seeded inputs from
``paper_2601_13776_amd.workloads`` (which holds no arithmetic of the method).

Modules
-------
bjorck   Frobenius pre-scaling and the Björck–Bowie iteration
         (Appendix A.5, "Björck–Bowie Iterative Projection").
aoc      RKO reshape, BCOP projector blocks, the block-convolution operator
         and the AOC kernel composition (Appendix B.1, eq. AOC = RKO ⊛ K_BCOP;
         stride / groups / dilation paragraphs of Appendix B.1).
conv     Circular convolution with stride, dilation and groups, its adjoint,
         the impulse-response Toeplitz matrix and the per-frequency FFT
         singular values (Section 4 and Appendix C, unit-testing scheme).
checks   Orthogonality deviation and norm ratios used as gates.
spectral Spectral pre-scaling by power iteration from a cached vector
         (Appendix A.5, Section 2), then Björck.
expo     Exponential map with spectral normalization (Appendix A.3) and the
         explicit conv exponential of Adaptive-SOC (Appendix B.2 theorem).
bjorck_grad  Vector-Jacobian product of pre-scaling + Björck (the
         derivative of the Appendix A.5 step, chained backwards).
aoc_grad Vector-Jacobian product of the composition (adjoint of each ⊛
         step, of the projector blocks and of P = V V^T).

Every function is pinned against closed forms, library routines (torch CPU
conv2d and conv_transpose2d, numpy SVD, scipy expm, torch.autograd), finite
differences or brute force: ``tests/test_oracle_pins.py``,
``tests/test_oracle_grad_pins.py``, ``tests/test_oracle_spectral_pins.py``,
``tests/test_oracle_expo_pins.py``; each module's docstring names its pins.
"""

from . import bjorck, aoc, conv, checks, bjorck_grad, aoc_grad, spectral, expo  # noqa: F401

__all__ = ["bjorck", "aoc", "conv", "checks", "bjorck_grad", "aoc_grad", "spectral", "expo"]
