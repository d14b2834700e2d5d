"""Host-side logic of bench.py on the CPU: the work counts behind its
rates (algorithmic and executed flops, checked against a direct count of
the tiles the kernels run), the CPU-baseline sample, the host report, the
traffic-record keying, and the refusal of more than one GPU."""

import hashlib
import os
import subprocess
import sys

import pytest

import bench
from paper_2601_13776_amd import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def tiles_counted(w, cls_name, big):
    """Executed flops by listing every tile: Gram tiles (i <= j) over the
    padded rows, update tiles over the padded columns (big: the matrices
    with N >= 1024 are on 256-tiles)."""
    shapes = [(max(r, c), min(r, c)) for r, c in w.matrix_shapes()]
    total = 0
    for m, n in shapes:
        if n <= 64 and m <= 128:
            continue
        b = 256 if (n >= 1024 and big) else 128
        if not cls_name.endswith(str(b)):
            continue
        mp, np_ = -(-m // b) * b, -(-n // b) * b
        for i in range(np_ // b):
            for j in range(np_ // b):
                if i <= j:
                    total += 2 * b * b * mp          # Gram tile (i, j): K = Mp
        total += (mp // b) * (np_ // b) * 2 * b * b * np_   # update tiles: K = Np
    return total * w.iters


@pytest.mark.parametrize("name,kernel,big", [("stress_4096x64_32x4096", "bjorck_bf16_256", True),
                                             ("imagenet_backbone25", "bjorck_bf16_128", False)])
def test_executed_flops_match_a_tile_count(name, kernel, big):
    w = wl.WORKLOADS[name]
    assert bench.executed_flops(w, kernel) == tiles_counted(w, kernel, big)


def _library_uses_256(shapes, vjp):
    """The library's own choice, read from its workspace sizes: the automatic
    choice sizes like the forced 256-tiles and unlike the forced 128."""
    import ctypes
    from paper_2601_13776_amd import orth
    L = orth.lib()
    sizes = []
    for tile in (0, 128, 256):
        opts = orth.orth_bjorck_opts(5, 0.5, 1, 1, 1, 1, 1, None, tile)
        n = ctypes.c_size_t()
        if vjp:
            arr = (orth.orth_vjp_mat * len(shapes))()
            for i, (r, c) in enumerate(shapes):
                b = 0x10000 + 0x4000000 * i
                arr[i] = orth.orth_vjp_mat(b, b + 0x1000000, b + 0x2000000, r, c, c, c, c)
            rc = L.orth_orthogonalize_vjp_workspace_size(arr, len(shapes), ctypes.byref(opts), ctypes.byref(n))
        else:
            arr = (orth.orth_mat * len(shapes))()
            for i, (r, c) in enumerate(shapes):
                b = 0x10000 + 0x4000000 * i
                arr[i] = orth.orth_mat(b, b + 0x2000000, r, c, c, c)
            rc = L.orth_orthogonalize_workspace_size(arr, len(shapes), ctypes.byref(opts), ctypes.byref(n))
        assert rc == 0
        sizes.append(n.value)
    assert sizes[1] != sizes[2]
    return sizes[0] == sizes[2]


@pytest.mark.parametrize("name", ["stress_4096x64_32x4096", "imagenet_backbone25"])
def test_bench_tile_rule_matches_the_library(name):
    shapes = wl.WORKLOADS[name].matrix_shapes()
    tall = [(max(r, c), min(r, c)) for r, c in shapes]
    assert bench.big_tiles(tall) == _library_uses_256(shapes, vjp=False) == _library_uses_256(shapes, vjp=True)


def test_stress_flop_counts():
    w = wl.WORKLOADS["stress_4096x64_32x4096"]
    n = 4096
    assert bench.class_flops(w, "bjorck_bf16_256") == 64 * 4 * n ** 3 * 25
    # the Gram computes 136 of 256 tiles: executed = (136 / 256 + 1) / 2 of the algorithmic
    assert bench.executed_flops(w, "bjorck_bf16_256") * 512 == bench.class_flops(w, "bjorck_bf16_256") * (136 + 256)


def test_cpu_sample_of_the_stress_batch():
    w = wl.WORKLOADS["stress_4096x64_32x4096"]
    by_shape, take = bench.cpu_sample(w)
    assert len(by_shape[(4096, 4096)]) == 64 and take[(4096, 4096)] == [by_shape[(4096, 4096)][0],
                                                                       by_shape[(4096, 4096)][-1]]
    assert take[(32, 32)] == by_shape[(32, 32)] and len(take[(32, 32)]) == 4096


def test_host_info():
    cores, model, blas = bench.host_info()
    assert cores == len(os.sched_getaffinity(0)) and cores >= 1
    assert isinstance(model, str) and model
    assert isinstance(blas, dict)


def test_traffic_record_keyed_to_sources(tmp_path, monkeypatch):
    """A record counts only for its kernel, workload and the exact sources it
    was measured on."""
    srcs = [tmp_path / "k.hip", tmp_path / "order.h"]
    for i, p in enumerate(srcs):
        p.write_text(f"source {i}\n")
    h = hashlib.sha256()
    for p in srcs:
        h.update(p.read_bytes())
    prof = tmp_path / "profiles"
    prof.mkdir()
    (prof / "traffic_kern_wl.md").write_text(
        f"text\n\n- kernel: kern\n- workload: wl\n- bytes_per_launch: 1234\n- source_sha256: {h.hexdigest()}\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "kernel_sources", lambda name: [str(p) for p in srcs])
    assert bench.measured_traffic("kern", "wl") == 1234
    assert bench.measured_traffic("kern", "other") is None
    srcs[0].write_text("changed\n")
    assert bench.measured_traffic("kern", "wl") is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=300, cwd=ROOT)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr) or "1 GPU" in (r.stdout + r.stderr), r.stdout + r.stderr
