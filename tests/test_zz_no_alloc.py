"""The allocation-free entry point (orth_orthogonalize_batched_noalloc,
through the C ABI) against the workspace entry point on the same inputs:
two calls in a row, the second on a smaller batch, so the second call runs
on the scratch the first one left behind.  Both entry points run the same
kernels on the same tables, so the outputs and statuses must agree bit for
bit."""

import numpy as np
import pytest
import torch

from paper_2601_13776_amd import orth
from paper_2601_13776_amd import workloads as wl

from gpu_util import DEV, to_dev

pytestmark = pytest.mark.gpu


def stored(seed, shapes, dtype="f32"):
    w = wl.Workload("noalloc", seed, dtype, 0, ())
    return [wl.stored_matrix(w, i, r, c) for i, (r, c) in enumerate(shapes)]


def both(st_list, iters, compute):
    ins = [to_dev(s) for s in st_list]
    ref = [torch.empty(t.shape, dtype=torch.float32, device=DEV) for t in ins]
    got = [torch.full(t.shape, float("nan"), dtype=torch.float32, device=DEV) for t in ins]
    s_ref = torch.full((len(ins),), -1, dtype=torch.int32, device=DEV)
    s_got = torch.full((len(ins),), -1, dtype=torch.int32, device=DEV)
    orth.orth_orthogonalize_batched(ins, ref, iters, compute=compute, status=s_ref)
    orth.orth_orthogonalize_batched_noalloc(ins, got, iters, compute=compute, status=s_got)
    torch.cuda.synchronize()
    assert torch.equal(s_ref, s_got)
    for a, b, s in zip(ref, got, st_list):
        assert torch.equal(a, b), s.shape
    return s_got.cpu().numpy()


@pytest.mark.parametrize("compute", ["f32", "bf16"])
def test_noalloc_matches_workspace_entry_point(compute):
    dtype = "bf16" if compute == "bf16" else "f32"
    # first call: small (fused kernel) and tiled matrices, tall and wide,
    # ragged; bf16 operands put the 1024-wide ones on 128-tiles
    first = [(512, 256), (256, 512), (300, 200), (1024, 1024), (64, 32), (32, 32), (100, 50), (129, 65)]
    print(f"[noalloc] {compute}: first call {len(first)} matrices", flush=True)
    status = both(stored(31, first, dtype), 12, compute)
    assert np.all(status == 0)
    # second call: fewer and smaller matrices on the scratch the first left
    second = [(200, 130), (40, 20), (96, 96)]
    print(f"[noalloc] {compute}: second call {len(second)} matrices", flush=True)
    status = both(stored(32, second, dtype), 9, compute)
    assert np.all(status == 0)


def test_noalloc_zero_matrix_and_statuses():
    """A zero matrix reports status 1 and outputs zeros, as with a
    workspace; the status array may also be left to the scratch."""
    st = stored(33, [(200, 100), (30, 30)])
    st[0][:] = 0
    status = both(st, 5, "f32")
    assert list(status) == [1, 0]
    ins = [to_dev(s) for s in st]
    outs = [torch.empty(t.shape, device=DEV) for t in ins]
    orth.orth_orthogonalize_batched_noalloc(ins, outs, 5)
    torch.cuda.synchronize()
    assert bool((outs[0] == 0).all())


def test_noalloc_rejects_a_batch_larger_than_its_scratch():
    # bf16 copies and E alone: 96 MiB (the fp32 output holds the iterate)
    ins = [torch.empty(4096, 4096, dtype=torch.bfloat16, device=DEV)]
    outs = [torch.empty(4096, 4096, device=DEV)]
    need = orth.orth_orthogonalize_workspace_size(ins, 10, compute="bf16", outs=outs)
    assert need > orth.ORTH_NOALLOC_SCRATCH_BYTES
    with pytest.raises(orth.OrthError) as e:
        orth.orth_orthogonalize_batched_noalloc(ins, outs, 10, compute="bf16")
    assert e.value.code == orth.ORTH_EWORKSPACE
    assert "holds" in str(e.value)


@pytest.mark.filterwarnings("ignore:The CUDA Graph is empty")
def test_noalloc_refuses_stream_capture():
    """Under HIP graph capture the allocation-free call refuses before it
    enqueues anything (its tables are copied from host memory of the call),
    and an ordinary call afterwards still matches the workspace entry point."""
    st = stored(34, [(300, 200), (40, 20)])
    ins = [to_dev(s) for s in st]
    outs = [torch.empty(t.shape, device=DEV) for t in ins]
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with pytest.raises(orth.OrthError) as e:
        with torch.cuda.graph(g):
            orth.orth_orthogonalize_batched_noalloc(ins, outs, 5)
    assert e.value.code == orth.ORTH_EUNSUPPORTED
    assert "captured" in str(e.value)
    torch.cuda.synchronize()
    status = both(st, 5, "f32")
    assert list(status) == [0, 0]
