"""GPU parity of the exponential parametrizations against the float64 oracle
(oracle/expo.py): the exponential map (orth_exp_map_batched) and the
explicit conv exponential (orth_conv_exp_batched).

Tolerances: relative Frobenius difference 1e-5 (fp32 products; the series
terms shrink by 1/k each step, so rounding stays at the level of one fp32
product of norm-1 matrices, ~1e-6); cached vectors 1e-5 (A = W - W^T is
formed in fp32 on the GPU, in fp64 by the oracle)."""

import math

import numpy as np
import pytest
import torch

from oracle import checks, conv, expo
from paper_2601_13776_amd import orth
from paper_2601_13776_amd import workloads as wl

from gpu_util import DEV, to_dev, to_f64

pytestmark = pytest.mark.gpu

REL = 1e-5


def stored(seed, shapes, dtype="f32"):
    w = wl.Workload("test", seed, dtype, 0, ())
    return [wl.stored_matrix(w, i, r, c) for i, (r, c) in enumerate(shapes)]


def run_exp(st, us, terms, q, out_dtype=torch.float32):
    ins = [to_dev(s) for s in st]
    outs = [torch.empty(t.shape, dtype=out_dtype, device=DEV) for t in ins]
    u = torch.from_numpy(np.concatenate(us).astype(np.float32)).to(DEV)
    status = torch.full((len(ins),), -1, dtype=torch.int32, device=DEV)
    orth.orth_exp_map_batched(ins, outs, terms, u, q, status=status)
    torch.cuda.synchronize()
    un = u.cpu().numpy()
    offs = np.cumsum([0] + [len(x) for x in us])
    return outs, [un[offs[i]:offs[i + 1]] for i in range(len(us))], status.cpu().numpy()


SIZES = [1, 2, 8, 33, 64, 130, 256]


@pytest.mark.parametrize("terms,q", [(12, 2), (6, 1)])
def test_exp_map_parity(terms, q):
    shapes = [(c, c) for c in SIZES]
    st = stored(801, shapes)
    rng = np.random.default_rng(802)
    us = [rng.standard_normal(c) for c in SIZES]
    outs, u_new, status = run_exp(st, us, terms, q)
    for s, u0, o, u1, c, stt in zip(st, us, outs, u_new, SIZES, status):
        ref, v = expo.exp_map(s.astype(np.float64), terms, u0.astype(np.float32).astype(np.float64), q)
        assert checks.relative_difference(to_f64(o), ref) <= REL, c
        if c > 1:
            assert stt == 0
            assert np.max(np.abs(u1 - v)) <= 1e-5, c
        else:
            assert stt == 1       # A = 0 for a 1 x 1 matrix: exp(0) = 1
    # 12 terms: orthogonal to fp32 rounding
    if terms == 12:
        for o in outs:
            g = to_f64(o)
            assert np.max(np.abs(g.T @ g - np.eye(g.shape[0]))) <= 1e-5


def test_exp_map_degenerate_and_bf16():
    shapes = [(16, 16), (16, 16), (40, 40)]
    st = stored(803, shapes, "bf16")
    sym = wl.as_f64(st[0])
    st[0] = wl.f32_to_bf16_bits((sym + sym.T).astype(np.float32))
    bad = wl.as_f64(st[1]).astype(np.float32)
    bad[2, 3] = np.nan
    st[1] = wl.f32_to_bf16_bits(bad)
    us = [np.ones(16), np.ones(16), np.linspace(-1, 1, 40)]
    outs, u_new, status = run_exp(st, us, 10, 2, torch.bfloat16)
    assert list(status) == [1, 2, 0]
    assert torch.equal(outs[0].float().cpu(), torch.eye(16))
    assert np.array_equal(u_new[0], np.ones(16, np.float32))
    assert torch.all(torch.isnan(outs[1].float()))
    ref, _ = expo.exp_map(wl.as_f64(st[2]), 10, us[2].astype(np.float32).astype(np.float64), 2)
    # bf16 output: one rounding of each element (u = 2^-9)
    assert checks.relative_difference(to_f64(outs[2]), ref) <= 1e-2


CONV_CASES = [  # c, k, terms, scale
    (4, 3, 4, 0.3), (16, 3, 6, 0.1), (32, 3, 8, 0.05), (6, 5, 3, 0.2), (8, 1, 10, 0.5), (64, 3, 5, 0.02),
    (3, 3, 1, 0.7),
]


def run_conv_exp(cases, dtype=torch.float32, seed=900):
    rng = np.random.default_rng(seed)
    layers, kerns = [], []
    for c, k, p, sc in cases:
        kern = rng.standard_normal((c, c, k, k)).astype(np.float32)
        if dtype == torch.bfloat16:
            kern = torch.from_numpy(kern).to(torch.bfloat16).float().numpy()
        kerns.append(kern)
        S = p * (k - 1) + 1
        layers.append(dict(kernel=torch.from_numpy(kern).to(DEV).to(dtype).contiguous(),
                           out=torch.full((c, c, S, S), float("nan"), dtype=dtype, device=DEV), terms=p, scale=sc))
    orth.orth_conv_exp_batched(layers)
    torch.cuda.synchronize()
    return layers, kerns


def test_conv_exp_parity_batched():
    layers, kerns = run_conv_exp(CONV_CASES)
    for (c, k, p, sc), L, kern in zip(CONV_CASES, layers, kerns):
        ref = expo.conv_exp(kern.astype(np.float64), p, sc)
        assert checks.relative_difference(to_f64(L["out"]), ref) <= REL, (c, k, p)


def test_conv_exp_bf16_storage():
    cases = [(16, 3, 5, 0.1), (8, 5, 3, 0.1)]
    layers, kerns = run_conv_exp(cases, torch.bfloat16, 901)
    for (c, k, p, sc), L, kern in zip(cases, layers, kerns):
        ref = expo.conv_exp(kern.astype(np.float64), p, sc)
        assert checks.relative_difference(to_f64(L["out"]), ref) <= 1e-2


def test_conv_exp_is_orthogonal_on_gpu():
    """A kernel scaled so that |conv(L)| <= 0.5: with 12 terms the explicit
    exponential preserves norms to the truncation bound (checked with the
    library's own norm check on random inputs)."""
    c, k, p, hw = 8, 3, 12, 16
    rng = np.random.default_rng(902)
    kern = rng.standard_normal((c, c, k, k))
    lk = expo.skew_kernel(kern)
    # |conv(L)| <= sum over taps of the spectral norms of the taps
    bound = sum(np.linalg.norm(lk[:, :, a, b], 2) for a in range(k) for b in range(k))
    scale = 0.5 / bound
    S = p * (k - 1) + 1
    L = dict(kernel=torch.from_numpy(kern.astype(np.float32)).to(DEV), out=torch.empty(c, c, S, S, device=DEV),
             terms=p, scale=scale)
    orth.orth_conv_exp_batched([L])
    x = torch.from_numpy(rng.standard_normal((4, c, hw, hw)).astype(np.float32)).to(DEV)
    ratio = orth.orth_check_norm_conv(L["out"], (c, c, S, 1, 1, 1), x)
    trunc = 0.5 ** (p + 1) * math.exp(0.5) / math.factorial(p + 1)
    assert float(torch.max(torch.abs(ratio - 1))) <= 1e-5 + trunc
    # and the explicit kernel reproduces the per-input series
    xs = to_f64(x)
    ref = xs.copy()
    term = xs.copy()
    lks = scale * lk
    for j in range(1, p + 1):
        term = conv.conv_circular(lks, term) / j
        ref = ref + term
    got = orth.orth_conv_apply(L["out"], (c, c, S, 1, 1, 1), x)
    assert checks.relative_difference(to_f64(got), ref) <= REL
