"""Seeded input generator: determinism, shapes, bf16 rounding."""

import numpy as np
import torch

from paper_2601_13776_amd import workloads as wl


def test_matrix_inventory_counts():
    counts = {name: len(wl.WORKLOADS[name].matrix_shapes()) for name in wl.WORKLOAD_ORDER}
    assert counts == {"conv3x3_c16": 5, "cifar_stack12": 54, "mixed_gds19": 229,
                      "imagenet_backbone25": 89, "stress_4096x64_32x4096": 4160}
    layers = {name: wl.WORKLOADS[name].n_layers for name in wl.WORKLOAD_ORDER}
    assert layers == {"conv3x3_c16": 1, "cifar_stack12": 12, "mixed_gds19": 19,
                      "imagenet_backbone25": 25, "stress_4096x64_32x4096": 4160}


def test_algorithmic_flops():
    f = {name: wl.algorithmic_bjorck_flops(wl.WORKLOADS[name].matrix_shapes(), wl.WORKLOADS[name].iters)
         for name in wl.WORKLOAD_ORDER}
    assert abs(f["cifar_stack12"] / 7.36e10 - 1) < 0.01
    assert abs(f["mixed_gds19"] / 4.35e10 - 1) < 0.01
    assert abs(f["imagenet_backbone25"] / 4.04e12 - 1) < 0.01
    assert abs(f["stress_4096x64_32x4096"] / 4.40e14 - 1) < 0.01


def test_deterministic_and_independent():
    w = wl.WORKLOADS["cifar_stack12"]
    a = wl.all_matrices(w)
    b = wl.all_matrices(w)
    assert wl.sha256_of(a) == wl.sha256_of(b)
    # one matrix regenerated on its own equals its place in the full list
    shapes = w.matrix_shapes()
    assert np.array_equal(wl.stored_matrix(w, 17, *shapes[17]), a[17])


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(100000) * np.exp(rng.uniform(-30, 30, 100000))).astype(np.float32)
    x[:4] = [0.0, -0.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8]      # ties to even
    ours = wl.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    back = wl.bf16_bits_to_f64(ours)
    assert np.array_equal(back, torch.from_numpy(x).to(torch.bfloat16).double().numpy())


def test_stress_rows():
    w = wl.WORKLOADS["stress_4096x64_32x4096"]
    m = wl.draw_matrix(w, 4100, 32, 32)
    norms = np.linalg.norm(m, axis=1)
    assert np.sum(norms > 20) == 2          # round(0.05 * 32) rows scaled by 100
