"""Helpers shared by the GPU tests: moving seeded inputs to the device and
calling the library through its binding.  No arithmetic of the method."""

import numpy as np
import torch

from paper_2601_13776_amd import orth
from paper_2601_13776_amd import workloads as wl

DEV = "cuda:0"


def to_dev(stored):
    """Stored matrix (float32 array or uint16 bf16 bits) -> device tensor."""
    if stored.dtype == np.uint16:
        return torch.from_numpy(stored.view(np.int16).copy()).view(torch.bfloat16).to(DEV)
    return torch.from_numpy(np.ascontiguousarray(stored)).to(DEV)


def to_f64(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def gpu_orthogonalize(stored_list, iters, compute="f32", out_dtype=torch.float32, beta=0.5, prescale="frobenius",
                      tile=0):
    ins = [to_dev(s) for s in stored_list]
    outs = [torch.empty(t.shape, dtype=out_dtype, device=DEV) for t in ins]
    status = torch.full((len(ins),), -1, dtype=torch.int32, device=DEV)
    orth.orth_orthogonalize_batched(ins, outs, iters, beta=beta, prescale=prescale, compute=compute,
                                    status=status, tile=tile)
    torch.cuda.synchronize()
    return outs, status.cpu().numpy()


def oracle_inputs(stored_list):
    return [wl.as_f64(s) for s in stored_list]


def random_geometries(seed, count, shapes_of):
    """Seeded random convolution geometries (cin, cout, k, stride, dilation,
    groups): k up to 5, stride up to 2, dilation up to 3, up to 4 groups and
    ragged channel counts; those that shapes_of (a parameter-shape rule that
    raises on an invalid geometry) refuses are drawn again."""
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < count:
        g = int(rng.choice([1, 1, 2, 3, 4]))
        geom = (g * int(rng.integers(2, 17)), g * int(rng.integers(1, 17)), int(rng.integers(1, 6)),
                int(rng.integers(1, 3)), int(rng.integers(1, 4)), g)
        try:
            shapes_of(*geom)
        except ValueError:
            continue
        out.append(geom)
    return out
