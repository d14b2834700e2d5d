"""Extreme shapes on the GPU: a dimension of 2^20 (the largest the
library accepts), aspect ratios up to 2^20 : 1 in both orientations, and
a 131072 x 1024 bf16 matrix on 256-tiles (Gram tiles over K = 131072).
The inputs are W = Q D with Q the first columns of a Householder
reflection and D diagonal (tests/reflected.py), whose Björck output is Q
times the oracle's iteration on D (App. A.5; pinned in
test_oracle_pins.py), so the reference costs O(rows x cols) at any size.
The GPU reads W rounded to its storage dtype while the reference starts
from the exact W: the iteration does not amplify that relative rounding
(D's values lie in [0.4, 1]), so the stated tolerances hold: 1e-5 with
fp32 products, 1e-2 with bf16 operands, whole matrix and (bf16) per
256 x 256 block."""

import numpy as np
import pytest
import torch

from oracle import bjorck, checks
from paper_2601_13776_amd import orth
from paper_2601_13776_amd import workloads as wl

import reflected
from gpu_util import DEV, to_f64

pytestmark = pytest.mark.gpu

REL_F32 = 1e-5
REL_BF16 = 1e-2
N_MAX = 1 << 20


def run(rows, cols, iters, compute, tile=0, seed=7):
    v, d = reflected.factors(seed, rows, cols)
    w = np.ascontiguousarray(reflected.matrix(v, d, rows, cols))
    if compute == "bf16":
        stored = wl.f32_to_bf16_bits(w.astype(np.float32))
        dev = torch.from_numpy(stored.view(np.int16)).view(torch.bfloat16).to(DEV)
    else:
        dev = torch.from_numpy(w.astype(np.float32)).to(DEV)
    del w
    out = torch.empty(dev.shape, dtype=torch.float32, device=DEV)
    status = torch.full((1,), -1, dtype=torch.int32, device=DEV)
    orth.orth_orthogonalize_batched([dev], [out], iters, compute=compute, status=status, tile=tile)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    ref = reflected.lift(v, bjorck.bjorck(np.diag(d), iters))
    return to_f64(out), (ref if rows >= cols else ref.T)


@pytest.mark.parametrize("rows,cols,iters", [(N_MAX, 1, 3), (1, N_MAX, 3), (1 << 18, 3, 6), (3, 1 << 18, 6)])
def test_extreme_aspect_f32(rows, cols, iters):
    print(f"[extremes] f32 {rows} x {cols}, T={iters}", flush=True)
    got, ref = run(rows, cols, iters, "f32")
    rel = checks.relative_difference(got, ref)
    print(f"[extremes]   relative {rel:.2e}", flush=True)
    assert rel <= REL_F32, rel


@pytest.mark.parametrize("rows,cols,iters,tile", [(N_MAX, 1, 3, 0), (1, N_MAX, 3, 0), (131072, 1024, 6, 256),
                                                   (1024, 65536, 6, 128)])
def test_extreme_shapes_bf16(rows, cols, iters, tile):
    print(f"[extremes] bf16 {rows} x {cols}, T={iters}, tile {tile}", flush=True)
    got, ref = run(rows, cols, iters, "bf16", tile=tile)
    rel = checks.relative_difference(got, ref)
    blocks = checks.tile_relative_differences(got, ref, 256) if min(rows, cols) > 1 else np.array([rel])
    print(f"[extremes]   relative {rel:.2e}, largest block {blocks.max():.2e}", flush=True)
    assert rel <= REL_BF16, rel
    assert blocks.max() <= REL_BF16, (blocks.max(), np.unravel_index(np.argmax(blocks), blocks.shape))
