"""Calls from several host threads at once (orthogonalization, its VJP and
the kernel composition), each thread on a stream of its own, so that the
library's shared host state (plan cache, pinned staging pool, per-thread
side streams and last errors) serves concurrent callers: every result must
be bit-identical to the same call made alone."""

import threading

import pytest
import torch

from paper_2601_13776_amd import orth
from paper_2601_13776_amd import workloads as wl

from gpu_util import DEV, to_dev

pytestmark = pytest.mark.gpu

# (name, seed, parameter dtype, shapes, compute, T, kind)
JOBS = [
    ("bf16 tiled", 31, "bf16", [(1024, 1024), (2048, 1024), (1100, 1030), (64, 32), (300, 700)], "bf16", 12, "fwd"),
    ("f32 mixed", 32, "f32", [(512, 256), (256, 256), (33, 17), (130, 64), (700, 300)], "f32", 10, "fwd"),
    ("bf16 small", 33, "bf16", [(32, 32)] * 200 + [(128, 64)] * 20, "bf16", 15, "fwd"),
    ("bf16 vjp", 34, "bf16", [(512, 512), (1024, 512), (64, 64), (200, 130)], "bf16", 8, "vjp"),
    # (cin, cout, k, stride, dilation, groups) of explicit kernels composed from given factors
    ("composition", 35, "f32",
     [(64, 64, 3, 1, 1, 1), (128, 256, 3, 2, 1, 1), (32, 32, 3, 1, 2, 4), (16, 32, 2, 2, 1, 2)], "f32", 0, "conv"),
]


def inputs(job):
    name, seed, dt, shapes = job[:4]
    if job[6] == "conv":
        gen = torch.Generator(device=DEV)
        gen.manual_seed(seed)
        layers = []
        for geom in shapes:
            rr, rc, npj, pr, pc = orth.orth_aoc_param_shapes(*geom)
            g = geom[5]
            layers.append(dict(geom=geom, rko=torch.randn(g, rr, rc, generator=gen, device=DEV),
                               proj=torch.randn(g, npj, pr, pc, generator=gen, device=DEV) if npj else None))
        return layers, None
    w = wl.Workload("threads", seed, dt, 0, ())
    ins = [to_dev(wl.stored_matrix(w, i, r, c)) for i, (r, c) in enumerate(shapes)]
    gen = torch.Generator(device=DEV)
    gen.manual_seed(seed)
    gouts = [torch.randn(s, generator=gen, device=DEV) for s in shapes]
    return ins, gouts


def run(job, ins, gouts):
    """One call of the job on the current stream; returns its outputs."""
    compute, iters, kind = job[4:]
    if kind == "conv":
        outs = []
        for L in ins:
            cin, cout, k, _, _, g = L["geom"]
            outs.append(torch.empty(cout, cin // g, k, k, device=DEV))
        orth.orth_build_conv_kernels_batched([dict(L, kernel=o) for L, o in zip(ins, outs)])
    elif kind == "fwd":
        outs = [torch.empty(t.shape, dtype=torch.float32, device=DEV) for t in ins]
        orth.orth_orthogonalize_batched(ins, outs, iters, compute=compute)
    else:
        outs = [torch.empty_like(t) for t in ins]
        orth.orth_orthogonalize_vjp_batched(ins, gouts, outs, iters, compute=compute)
    return outs


def test_concurrent_callers_match_single_calls():
    data = [inputs(job) for job in JOBS]
    torch.cuda.synchronize()
    alone = [run(job, *d) for job, d in zip(JOBS, data)]
    torch.cuda.synchronize()
    reps = 4
    results = [None] * len(JOBS)
    errors = []
    start = threading.Barrier(len(JOBS))

    def worker(k):
        try:
            stream = torch.cuda.Stream(device=DEV)
            with torch.cuda.stream(stream):
                start.wait()
                results[k] = [run(JOBS[k], *data[k]) for _ in range(reps)]
            stream.synchronize()
        except Exception as e:   # surfaced in the main thread
            errors.append((JOBS[k][0], repr(e)))

    threads = [threading.Thread(target=worker, args=(k,)) for k in range(len(JOBS))]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads), "a caller thread did not finish"
    assert not errors, errors
    torch.cuda.synchronize()
    for job, ref, got in zip(JOBS, alone, results):
        print(f"[threads] {job[0]}: {len(got)} calls", flush=True)
        for r in range(reps):
            for i, (a, b) in enumerate(zip(got[r], ref)):
                assert torch.equal(a, b), (job[0], r, i)


def test_timing_from_concurrent_callers():
    """Per-kernel timing with the callers on four threads and streams: the
    same launches counted as when the calls run one after another, every
    event pair complete (each launch's end pairs with its start on its own
    stream), and the covered span no longer than the summed durations."""
    data = [inputs(job) for job in JOBS]
    torch.cuda.synchronize()

    def counts():
        names = orth.orth_timing_names()
        return {n: orth.orth_timing_read(n) for n in names}

    orth.orth_timing_reset()
    orth.orth_timing_enable(True)
    try:
        for job, d in zip(JOBS, data):
            run(job, *d)
        torch.cuda.synchronize()
        alone = counts()
        orth.orth_timing_reset()
        errors = []
        start = threading.Barrier(len(JOBS))

        def worker(k):
            try:
                stream = torch.cuda.Stream(device=DEV)
                with torch.cuda.stream(stream):
                    start.wait()
                    run(JOBS[k], *data[k])
                stream.synchronize()
            except Exception as e:
                errors.append((JOBS[k][0], repr(e)))

        threads = [threading.Thread(target=worker, args=(k,)) for k in range(len(JOBS))]
        for t in threads:
            t.start()
        for t in threads:
            t.join(timeout=120)
        assert not any(t.is_alive() for t in threads) and not errors, errors
        torch.cuda.synchronize()
        together = counts()
        prefixes = sorted({n.split("_")[0] for n in together})
        span_ms, span_n = orth.orth_timing_span(*prefixes)
    finally:
        orth.orth_timing_enable(False)
        orth.orth_timing_reset()
    assert {n: c[1] for n, c in together.items()} == {n: c[1] for n, c in alone.items()}
    assert all(c[0] > 0 for c in together.values())
    assert span_n == sum(c[1] for c in together.values())
    assert 0 < span_ms <= sum(c[0] for c in together.values()) * (1 + 1e-6)
