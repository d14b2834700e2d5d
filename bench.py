"""Benchmark of one parametrization step on one MI355X.

A step orthogonalizes every free matrix of a workload in one batched call
(orth_orthogonalize_batched) and builds every conv kernel in one batched call
(orth_build_conv_kernels_batched).  Inputs are seeded synthetic parameters
already resident in HBM.  Prints one JSON line.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                    [--no-cpu-baseline] [--vjp [--vjp-steps K]] [--copy-calibration]
                    [--prescale spectral [--power-iters Q]] [--iters T]
                    [--conv-apply [--apply-batch B]] [--expo]

With --vjp the backward pass (dL/dK and dL/d(output) back to the raw
parameters) is timed too and reported under "vjp".
"""

import argparse
import concurrent.futures as cf
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2601_13776_amd import workloads as wl  # noqa: E402

PEAK_BF16_TFLOPS = 2516.6   # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3     # MI355X fp32 MFMA
PEAK_HBM_GBS = 8000.0
METRIC = "orthogonalized layers/sec per param step; Björck TFLOP/s as % MFMA peak"
DEFAULT_WORKLOAD = "stress_4096x64_32x4096"


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def make_inputs(w, torch, dev):
    shapes = w.matrix_shapes()

    def one(i):
        return wl.stored_matrix(w, i, *shapes[i])

    tensors = [None] * len(shapes)
    with cf.ThreadPoolExecutor(max_workers=8) as ex:
        for i, s in zip(range(len(shapes)), ex.map(one, range(len(shapes)))):
            if s.dtype == np.uint16:
                t = torch.from_numpy(s.view(np.int16)).view(torch.bfloat16)
            else:
                t = torch.from_numpy(s)
            tensors[i] = t.to(dev, non_blocking=False)
    return tensors


def allocate_outputs(w, ins, torch, dev, out_dtype):
    """Output tensors for every matrix.  The factors of a conv layer are views
    into that layer's contiguous RKO / projector buffers, so the batched
    orthogonalization writes them exactly where the kernel build reads them."""
    outs = [None] * len(ins)
    layers = []
    for layer, (a, b) in zip(w.layers, wl.layer_matrix_ranges(w)):
        if not isinstance(layer, wl.ConvLayer):
            for i in range(a, b):
                outs[i] = torch.empty(ins[i].shape, dtype=out_dtype, device=dev)
            continue
        g, npj = layer.groups, layer.n_proj
        per = 1 + npj
        rr, rc = ins[a].shape
        rko = torch.empty(g, rr, rc, device=dev, dtype=out_dtype)
        proj = torch.empty(g, npj, layer.c, layer.c // 2, device=dev, dtype=out_dtype) if npj else None
        for j in range(g):
            outs[a + j * per] = rko[j]
            for t in range(npj):
                outs[a + j * per + 1 + t] = proj[j, t]
        kern = torch.empty(layer.cout, layer.c, layer.k, layer.k, device=dev, dtype=out_dtype)
        layers.append(dict(geom=(layer.cin, layer.cout, layer.k, layer.stride, layer.dilation, layer.groups),
                           rko=rko, proj=proj, kernel=kern))
    return outs, layers


# traffic records: profiles/traffic_<kernel>_<workload>.md
# the traffic depends on the kernel and on the tile order the host planner builds
def kernel_sources(kernel_name):
    """Sources whose change invalidates a traffic record: the kernel and the
    planner code that orders its tiles."""
    files = ("bjorck_bf16.hip", "tile_order.h") if "bf16" in kernel_name else ("gemm_f32.hip", "host.hip")
    return [os.path.join(ROOT, "paper_2601_13776_amd", "csrc", f) for f in files]


def measured_traffic(kernel_name, workload):
    """HBM bytes per launch of the dominant kernel from the committed
    rocprofv3 FETCH_SIZE / WRITE_SIZE measurement, or None when there is none
    for this kernel and workload or the kernel or planner source changed
    since."""
    import hashlib
    import re
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel_name}_{workload}.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    fields = dict(re.findall(r"^- (\w+): (\S+)$", text, flags=re.M))
    try:
        h = hashlib.sha256()
        for f in kernel_sources(kernel_name):
            h.update(open(f, "rb").read())
        src_hash = h.hexdigest()
        if fields.get("kernel") != kernel_name or fields.get("workload") != workload \
                or fields.get("source_sha256") != src_hash:
            return None
        return int(fields["bytes_per_launch"])
    except (KeyError, ValueError, OSError):
        return None


def big_tiles(shapes):
    """The library's choice of 256-tiles for the matrices with N >= 1024 (a
    tall list of (M, N)): their update tiles of 256 fill four waves of the
    256 compute units."""
    return sum(-(-m // 256) * -(-n // 256) for m, n in shapes if n >= 1024) >= 4 * 256


def class_flops(w, kernel_name):
    """Algorithmic Björck flops of one parametrization step that run in the
    named tiled kernel: every matrix of its size class contributes
    4 m n min(m, n) T (a Gram and an update product per iteration)."""
    out = 0
    shapes = [(max(r, c), min(r, c)) for r, c in w.matrix_shapes()]
    big = big_tiles(shapes)
    for m, n in shapes:
        if n <= 64 and m <= 128:          # fused small-matrix kernel
            continue
        if w.dtype == "bf16":
            cls = "256" if n >= 1024 and big else "128"
            if not kernel_name.endswith(cls):
                continue
        out += 4 * m * n * n * w.iters
    return out


def executed_flops(w, kernel_name, iters=None):
    """Flops the MFMA pipes execute in the named tiled Björck kernel per
    parametrization step: a Gram launch computes only the upper tiles of the
    symmetric E = I - X^T X (tn (tn + 1) / 2 tiles of B x B over Mp), an
    update launch every tile of X E (tm tn tiles over Np), both on the tile
    grid the planner pads to.  The algorithmic count (class_flops) charges
    the dense 2 m n^2 for the Gram instead."""
    T = w.iters if iters is None else iters
    shapes = [(max(r, c), min(r, c)) for r, c in w.matrix_shapes()]
    big = big_tiles(shapes)
    out = 0
    for m, n in shapes:
        if n <= 64 and m <= 128:
            continue
        if w.dtype == "bf16":
            cls = 256 if n >= 1024 and big else 128
            if not kernel_name.endswith(str(cls)):
                continue
        else:
            cls = 64
        mp, np_ = -(-m // cls) * cls, -(-n // cls) * cls
        tm, tn = mp // cls, np_ // cls
        out += T * (tn * (tn + 1) // 2 * 2 * cls * cls * mp + tm * tn * 2 * cls * cls * np_)
    return out


def vjp_flops(w):
    """Algorithmic flops of one vector-Jacobian product of the whole
    workload: the forward recomputation (a Gram and an update product per
    step, the last update skipped: (4T - 2) m n^2) and the gradient
    recurrence (X^T Y, Y E and X S per step: 6 T m n^2)."""
    out = 0
    for r, c in w.matrix_shapes():
        m, n = max(r, c), min(r, c)
        out += (10 * w.iters - 2) * m * n * n
    return out


def run_vjp(w, ins, outs, layers, status, compute, steps, warmup, torch, orth, dev):
    """Time steps of the backward pass: dL/dK -> factor gradients for every
    conv layer (composition VJP), then dL/d(factor) -> dL/d(raw parameter)
    for every matrix (Björck VJP).  Upstream gradients are seeded N(0, 1)."""
    gen = torch.Generator(device=dev)
    gen.manual_seed(w.seed + 200)
    gouts = [torch.randn(o.shape, generator=gen, device=dev, dtype=torch.float32) for o in outs]
    gins = [torch.empty_like(t) for t in ins]
    vlayers = []
    for L in layers:
        gk = torch.randn(L["kernel"].shape, generator=gen, device=dev, dtype=L["kernel"].dtype)
        vlayers.append(dict(geom=L["geom"], rko=L["rko"], proj=L["proj"], grad_kernel=gk,
                            grad_rko=torch.empty_like(L["rko"]),
                            grad_proj=torch.empty_like(L["proj"]) if L["proj"] is not None else None))
    # the conv factors' upstream gradients are the composition VJP's outputs
    k = 0
    for layer, (a, b) in zip(w.layers, wl.layer_matrix_ranges(w)):
        if not isinstance(layer, wl.ConvLayer):
            continue
        V = vlayers[k]
        k += 1
        per = 1 + layer.n_proj
        for j in range(layer.groups):
            gouts[a + j * per] = V["grad_rko"][j]
            for t in range(layer.n_proj):
                gouts[a + j * per + 1 + t] = V["grad_proj"][j, t]
    bws = orth.orth_orthogonalize_vjp_batched(ins, gouts, gins, w.iters, compute=compute, status=status)
    cws = orth.orth_build_conv_kernels_vjp_batched(vlayers) if vlayers else None
    torch.cuda.synchronize()
    log(f"[bench] vjp workspace {bws.numel() / 2**30:.2f} GiB")

    def vstep():
        if vlayers:
            orth.orth_build_conv_kernels_vjp_batched(vlayers, workspace=cws)
        orth.orth_orthogonalize_vjp_batched(ins, gouts, gins, w.iters, compute=compute, status=status,
                                            workspace=bws)

    for i in range(warmup):
        vstep()
        torch.cuda.synchronize()
        log(f"[bench] vjp warmup {i + 1}/{warmup}")
    # events only around the GEMM-chain launches (each timed launch costs a
    # few microseconds of stream time)
    orth.orth_timing_filter("bjorck_", "vjp_fwd_", "vjp_s_", "vjp_update_")
    orth.orth_timing_enable(True)
    orth.orth_timing_reset()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        vstep()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    log(f"[bench] vjp timed {steps} steps")
    names = orth.orth_timing_names()
    kt = {n: orth.orth_timing_read(n) for n in names}
    # wall time covered by the GEMM-chain launches (side streams overlap)
    gemm_ms = orth.orth_timing_span("bjorck_", "vjp_fwd_", "vjp_s_", "vjp_update_")[0] / steps
    orth.orth_timing_enable(False)
    orth.orth_timing_filter()
    ms = (t1 - t0) * 1e3 / steps
    flops = vjp_flops(w)
    peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS
    # roofline of the dominant gradient-recurrence kernel: its class's
    # algorithmic 6 m n^2 T flops per step over its measured time
    cands = [n for n in names if n.startswith("bjorck_vjp_bf16") or n in ("vjp_s_f32", "vjp_update_f32")]
    roof = None
    if cands:
        dom = max(cands, key=lambda n: kt[n][0])
        tot_ms, launches = kt[dom]
        cf_ = class_flops(w, dom[len("bjorck_vjp"):] if dom.startswith("bjorck_vjp") else "") * 6 // 4 * steps
        if not dom.startswith("bjorck_vjp"):   # fp32: S and update launches timed apart, each half
            cf_ = (vjp_class_flops_f32(w) * steps) // 2
        ach = cf_ / (tot_ms / 1e3) / 1e12
        roof = {"bound": "mfma", "kernel": dom, "achieved": round(ach, 1), "peak": peak, "unit": "TFLOP/s",
                "frac": round(ach / peak, 4), "traffic": measured_traffic(dom, w.name),
                "avg_launch_ms": round(tot_ms / launches, 4),
                "algorithmic_flops_per_launch": int(cf_ / launches)}
    # The training pattern: a parametrization step that keeps its iterates
    # and tap grids in the VJP workspaces (orth_orthogonalize_save_batched,
    # orth_build_conv_kernels_save_batched) and VJPs that reuse them instead
    # of recomputing the forward steps.
    klayers = [dict(geom=L["geom"], rko=L["rko"], proj=L["proj"], kernel=L["kernel"]) for L in layers]

    def save_step():   # the parametrization step, keeping what the VJP needs
        orth.orth_orthogonalize_save_batched(ins, outs, w.iters, compute=compute, status=status, workspace=bws)
        if klayers:
            orth.orth_build_conv_kernels_save_batched(klayers, workspace=cws)

    def saved_step():
        if vlayers:
            orth.orth_build_conv_kernels_vjp_batched(vlayers, workspace=cws, saved=True)
        orth.orth_orthogonalize_vjp_batched(ins, gouts, gins, w.iters, compute=compute, status=status,
                                            workspace=bws, saved=True)

    save_step()
    saved_step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        save_step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for _ in range(steps):
        saved_step()
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    log(f"[bench] saving forward and saved vjp timed {steps} steps each")
    save_ms = (t1 - t0) * 1e3 / steps
    saved_ms = (t2 - t1) * 1e3 / steps
    return {"ms_per_step": round(ms, 3), "layers_per_s": round(w.n_layers / (ms / 1e3), 3),
            "algorithmic_flops_per_step": flops,
            "tflops_algorithmic": round(flops / (ms / 1e3) / 1e12, 1),
            "gemm_tflops_algorithmic": round(flops / (gemm_ms / 1e3) / 1e12, 1) if gemm_ms > 0 else None,
            "gemm_pct_peak": round(100 * flops / (gemm_ms / 1e3) / 1e12 / peak, 2) if gemm_ms > 0 else None,
            "kernel_ms_per_step": {n: round(kt[n][0] / steps, 4) for n in names},
            "roofline": roof,
            "saved": {"save_forward_ms": round(save_ms, 3), "vjp_ms_per_step": round(saved_ms, 3),
                      "train_step_ms": round(save_ms + saved_ms, 3)}}


def vjp_class_flops_f32(w):
    """Gradient-recurrence flops (6 m n^2 T) of the matrices that run on the
    fp32 tile GEMM (every matrix with fp32 products, the small bucket with
    bf16 products)."""
    out = 0
    for r, c in w.matrix_shapes():
        m, n = max(r, c), min(r, c)
        if w.dtype == "bf16" and not (n <= 64 and m <= 128):
            continue
        out += 6 * m * n * n * w.iters
    return out


def vjp_cpu_baseline(w, budget_s=25.0):
    """Time the float64 oracle VJP on a bounded sample: per shape, one matrix
    (up to 64 for small shapes) at T = 2, scaled to the workload's T by the
    (10 T - 2) algorithmic step count and to all matrices by count."""
    from oracle import bjorck_grad
    shapes = w.matrix_shapes()
    by_shape = {}
    for i, s in enumerate(shapes):
        by_shape.setdefault(s, []).append(i)
    rng = np.random.default_rng(7)
    per_shape, desc = {}, []
    t_start = time.perf_counter()
    t_s = 2
    for s, idx in sorted(by_shape.items(), key=lambda kv: kv[0][0] * kv[0][1]):
        n_take = 1 if s[0] * s[1] >= 512 * 512 else min(len(idx), 64)
        y = rng.standard_normal(s)
        t0 = time.perf_counter()
        for i in idx[:n_take]:
            bjorck_grad.bjorck_vjp(wl.as_f64(wl.stored_matrix(w, i, *s)), y, t_s)
        per_shape[s] = (time.perf_counter() - t0) / n_take * (10 * w.iters - 2) / (10 * t_s - 2)
        desc.append(f"{n_take}x{s[0]}x{s[1]}")
        if time.perf_counter() - t_start > budget_s:
            break
    ref_s = max(per_shape, key=lambda s: s[0] * s[1] * min(s))
    ref_f = ref_s[0] * ref_s[1] * min(ref_s)
    total = sum(per_shape.get(s, per_shape[ref_s] * s[0] * s[1] * min(s) / ref_f) * len(idx)
                for s, idx in by_shape.items())
    cores, model, blas = host_info()
    return {"value": w.n_layers / total, "unit": "layers/s", "cores": cores, "kind": "oracle",
            "cpu_model": model, "blas": blas,
            "sample": f"float64 numpy oracle VJP (Björck only), timed {'+'.join(desc)} at T={t_s} and scaled to "
                      f"T={w.iters} by (10T-2) and by matrix count (estimated full backward {total:.1f} s)",
            "est_step_s": total}


# input resolution of the first conv layer of each workload (halved after
# every stride-2 layer; the ImageNet-like widths 128..1024 run at 56..7)
APPLY_HW = {"conv3x3_c16": 16, "cifar_stack12": 32, "mixed_gds19": 32, "imagenet_backbone25": 56}


def run_conv_apply(w, layers, batch, steps, torch, orth, dev):
    """Time the forward and the transposed application of every conv layer's
    explicit kernel to a batch of images; algorithmic flop
    2 B (H/s)(W/s) cout (cin/g) k^2 per layer and direction."""
    hw = APPLY_HW.get(w.name)
    if not layers or hw is None:
        return None
    gen = torch.Generator(device=dev)
    gen.manual_seed(w.seed + 400)
    jobs = []
    prev_c = None
    for L in layers:
        cin, cout, k, s, d, g = L["geom"]
        if w.name == "imagenet_backbone25" and prev_c is not None and cin != prev_c:
            hw //= 2
        prev_c = cout
        x = torch.randn(batch, cin, hw, hw, generator=gen, device=dev)
        yt = torch.randn(batch, cout, hw // s, hw // s, generator=gen, device=dev)
        flops = 2 * batch * (hw // s) ** 2 * cout * (cin // g) * k * k
        jobs.append((L, x, yt, flops))
        hw //= s
    def one():
        for L, x, yt, _ in jobs:
            orth.orth_conv_apply(L["kernel"], L["geom"], x)
            orth.orth_conv_apply(L["kernel"], L["geom"], yt, transposed=True)
    one()
    torch.cuda.synchronize()
    orth.orth_timing_filter("conv_apply")
    orth.orth_timing_enable(True)
    orth.orth_timing_reset()
    t0 = time.perf_counter()
    for _ in range(steps):
        one()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    kt = {n: orth.orth_timing_read(n) for n in ("conv_apply", "conv_apply_transposed")}
    orth.orth_timing_enable(False)
    orth.orth_timing_filter()
    flops = sum(j[3] for j in jobs)
    out = {"batch": batch, "first_layer_hw": APPLY_HW[w.name], "ms_per_pass": round((t1 - t0) * 1e3 / steps, 3),
           "algorithmic_flops_per_direction": flops}
    for n, key in (("conv_apply", "forward"), ("conv_apply_transposed", "transposed")):
        ms = kt[n][0] / steps
        ach = flops / (ms / 1e3) / 1e12
        out[key] = {"ms": round(ms, 3), "roofline": {"bound": "mfma", "kernel": n, "achieved": round(ach, 1),
                                                     "peak": PEAK_F32_TFLOPS, "unit": "TFLOP/s",
                                                     "frac": round(ach / PEAK_F32_TFLOPS, 4), "traffic": None,
                                                     "avg_launch_ms": round(kt[n][0] / kt[n][1], 4)}}
    return out


def run_expo(w, ins, steps, torch, orth, dev, terms=12, conv_terms=6):
    """Exponential map of every square matrix of the workload and explicit
    conv exponential of every stride-1 c -> c conv layer; algorithmic flop:
    (p - 1) 2 C^3 per matrix, and 2 c^3 per tap product of the conv series."""
    sq = [t for t in ins if t.shape[0] == t.shape[1] and t.shape[0] > 1]
    convs = [L for L in w.layers if hasattr(L, "k") and L.stride == 1 and L.cin == L.cout and L.groups == 1
             and L.k % 2 == 1]
    out = {}
    gen = torch.Generator(device=dev)
    gen.manual_seed(w.seed + 500)
    jobs = []
    if sq:
        outs = [torch.empty(t.shape, dtype=torch.float32, device=dev) for t in sq]
        u = torch.randn(sum(t.shape[0] for t in sq), generator=gen, device=dev)
        ws = orth.orth_exp_map_batched(sq, outs, terms, u, 1)
        flops = sum((terms - 1) * 2 * t.shape[0] ** 3 for t in sq)
        jobs.append(("exp_map", lambda: orth.orth_exp_map_batched(sq, outs, terms, u, 1, workspace=ws), flops,
                     "exp_map_series", len(sq)))
    if convs:
        layers = []
        flops = 0
        for L in convs:
            c, k = L.cin, L.k
            S = conv_terms * (k - 1) + 1
            kern = torch.randn(c, c, k, k, generator=gen, device=dev)
            layers.append(dict(kernel=kern, out=torch.empty(c, c, S, S, device=dev), terms=conv_terms, scale=0.1))
            for j in range(2, conv_terms + 1):
                sp, sj = (j - 1) * (k - 1) + 1, j * (k - 1) + 1
                pairs = sum(1 for y in range(sj) for x in range(sj) for r in range(k) for t in range(k)
                            if 0 <= y - r < sp and 0 <= x - t < sp)
                flops += pairs * 2 * c ** 3
        cws = orth.orth_conv_exp_batched(layers)
        jobs.append(("conv_exp", lambda: orth.orth_conv_exp_batched(layers, workspace=cws), flops,
                     "conv_exp_series", len(layers)))
    torch.cuda.synchronize()
    for name, fn, flops, kname, count in jobs:
        fn()
        torch.cuda.synchronize()
        orth.orth_timing_filter(kname)
        orth.orth_timing_enable(True)
        orth.orth_timing_reset()
        t0 = time.perf_counter()
        for _ in range(steps):
            fn()
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        kt = orth.orth_timing_read(kname)
        orth.orth_timing_enable(False)
        orth.orth_timing_filter()
        ms = (t1 - t0) * 1e3 / steps
        kms = kt[0] / steps
        ach = flops / (kms / 1e3) / 1e12
        out[name] = {"count": count, "terms": terms if name == "exp_map" else conv_terms,
                     "ms_per_call": round(ms, 3), "algorithmic_flops": flops,
                     "roofline": {"bound": "mfma", "kernel": kname, "achieved": round(ach, 1),
                                  "peak": PEAK_F32_TFLOPS, "unit": "TFLOP/s", "frac": round(ach / PEAK_F32_TFLOPS, 4),
                                  "traffic": None, "avg_launch_ms": round(kt[0] / kt[1], 4)}}
    return out or None


def host_info():
    """Cores this process may run on, the CPU model and the BLAS library
    (name, version, threads) that NumPy calls."""
    model = platform.processor() or platform.machine()
    try:
        fields = {}
        with open("/proc/cpuinfo") as f:
            for line in f:
                if not line.strip():
                    break          # the first processor's block
                k, _, v = line.partition(":")
                fields[k.strip()] = v.strip()
        if "model name" in fields:
            # a virtualized host may report only the vendor line; the family
            # and model numbers still name the part
            model = fields["model name"]
            if "cpu family" in fields and "model" in fields:
                model += f" (family {fields['cpu family']}, model {fields['model']})"
    except OSError:
        pass
    blas = {}
    try:
        from threadpoolctl import threadpool_info
        for i in threadpool_info():
            if i.get("user_api") == "blas":
                blas = {"library": i.get("internal_api"), "version": i.get("version"),
                        "threads": i.get("num_threads"), "file": os.path.basename(i.get("filepath", ""))}
                break
    except Exception:  # pragma: no cover
        pass
    return len(os.sched_getaffinity(0)), model, blas


def cpu_sample(w):
    """The matrices the CPU legs time, per shape: for the stress batch two
    of the 64 4096^2 matrices (0 and 63) and all 4096 32^2 ones; otherwise
    every matrix of shapes up to 1024 x 1024 and two of each larger shape."""
    shapes = w.matrix_shapes()
    by_shape = {}
    for i, s_ in enumerate(shapes):
        by_shape.setdefault(s_, []).append(i)
    take = {}
    for s_, idx in by_shape.items():
        take[s_] = idx if s_[0] * s_[1] <= 1024 * 1024 else [idx[0], idx[-1]] if len(idx) > 1 else idx
    return by_shape, take


def plain_f32_bjorck(w32, iters, beta=0.5):
    """The Björck step (App. A.5) in plain NumPy float32 (BLAS sgemm),
    Frobenius pre-scaling, smaller Gram: the 'plain CPU fp32' baseline."""
    x = w32 if w32.shape[0] >= w32.shape[1] else w32.T
    x = x / np.float32(np.sqrt(np.sum(x * x, dtype=np.float64)))
    b = np.float32(beta)
    for _ in range(iters):
        x = (1 + b) * x - b * (x @ (x.T @ x))
    return x if w32.shape[0] >= w32.shape[1] else x.T


def cpu_baseline(w):
    """Time the float64 oracle (and a plain float32 NumPy run of the same
    formula) on a bounded sample of the workload, scaled by matrix count to
    the whole Björck step (labelled extrapolated when a shape was sampled)."""
    from oracle import bjorck
    cores, model, blas = host_info()
    by_shape, take = cpu_sample(w)
    per64, per32, desc = {}, {}, []
    extrapolated = False
    for s_, idx in sorted(by_shape.items(), key=lambda kv: kv[0][0] * kv[0][1]):
        sel = take[s_]
        mats = [wl.as_f64(wl.stored_matrix(w, i, *s_)) for i in sel]
        t0 = time.perf_counter()
        for m in mats:
            bjorck.bjorck(m, w.iters)
        per64[s_] = (time.perf_counter() - t0) / len(sel)
        m32 = [m.astype(np.float32) for m in mats]
        t0 = time.perf_counter()
        for m in m32:
            plain_f32_bjorck(m, w.iters)
        per32[s_] = (time.perf_counter() - t0) / len(sel)
        desc.append(f"{len(sel)}/{len(idx)}x{s_[0]}x{s_[1]}")
        extrapolated |= len(sel) < len(idx)
    tot64 = sum(per64[s_] * len(idx) for s_, idx in by_shape.items())
    tot32 = sum(per32[s_] * len(idx) for s_, idx in by_shape.items())
    label = "extrapolated by matrix count" if extrapolated else "every matrix timed"
    return {"value": w.n_layers / tot64, "unit": "layers/s", "cores": cores, "kind": "oracle",
            "sample": f"float64 NumPy oracle, Björck T={w.iters} with Frobenius pre-scaling of the workload's "
                      f"matrices: timed {'+'.join(desc)} (timed/total x shape), {label} to the whole "
                      f"{len(w.matrix_shapes())}-matrix step ({tot64:.1f} s)",
            "est_step_s": float(f"{tot64:.4g}"), "cpu_model": model, "blas": blas,
            "plain_cpu_fp32": {"value": w.n_layers / tot32, "unit": "layers/s", "est_step_s": float(f"{tot32:.4g}"),
                               "kind": "plain NumPy float32 (BLAS sgemm), same formula and sample"}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD, choices=wl.WORKLOAD_ORDER)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--prescale", default="frobenius", choices=["frobenius", "spectral"],
                    help="spectral: power iteration from cached vectors (warmed once before timing)")
    ap.add_argument("--power-iters", type=int, default=1)
    ap.add_argument("--iters", type=int, default=None, help="override the workload's Björck step count")
    ap.add_argument("--conv-apply", action="store_true",
                    help="also time the application of every conv layer's kernel (forward and transposed) "
                         "to a batch of images")
    ap.add_argument("--apply-batch", type=int, default=64)
    ap.add_argument("--expo", action="store_true",
                    help="also time the exponential map of every square matrix (12 terms) and the explicit conv "
                         "exponential of every stride-1 c -> c conv layer (6 terms)")
    ap.add_argument("--vjp", action="store_true",
                    help="also time the backward pass (composition and Björck vector-Jacobian products)")
    ap.add_argument("--vjp-steps", type=int, default=3)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run one plain 1 GiB device copy (for HBM counter scaling)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(the independent matrices would be distributed across GPUs by size)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2601_13776_amd import orth

    if not os.path.exists(orth._LIB_PATH):
        from paper_2601_13776_amd import build
        build.build()
    dev = torch.device("cuda:0")
    w = wl.WORKLOADS[args.workload]
    if args.iters is not None:
        import dataclasses
        w = dataclasses.replace(w, iters=args.iters)
    log(f"[bench] generating {w.name}: {len(w.matrix_shapes())} matrices")
    ins = make_inputs(w, torch, dev)
    out_dtype = torch.float32
    outs, layers = allocate_outputs(w, ins, torch, dev, out_dtype)
    status = torch.zeros(len(ins), dtype=torch.int32, device=dev)
    compute = "bf16" if w.dtype == "bf16" else "f32"
    pkw = {}
    if args.prescale == "spectral":
        # cached vectors warmed by a few power steps, as after earlier parameter updates
        gen = torch.Generator(device=dev)
        gen.manual_seed(w.seed + 300)
        u = torch.randn(sum(min(t.shape) for t in ins), generator=gen, device=dev)
        orth.orth_orthogonalize_batched(ins, outs, 0, compute=compute, status=status, prescale="spectral",
                                        power_iters=5, u=u)
        pkw = dict(prescale="spectral", power_iters=args.power_iters, u=u)
    ws = orth.orth_orthogonalize_batched(ins, outs, w.iters, compute=compute, status=status, **pkw)
    conv_ws = None
    torch.cuda.synchronize()
    log(f"[bench] workspace {ws.numel() / 2**30:.2f} GiB")

    def step():
        nonlocal conv_ws
        orth.orth_orthogonalize_batched(ins, outs, w.iters, compute=compute, status=status, workspace=ws, **pkw)
        if layers:
            conv_ws = orth.orth_build_conv_kernels_batched(layers, workspace=conv_ws)

    for i in range(args.warmup):
        step()
        torch.cuda.synchronize()
        log(f"[bench] warmup {i + 1}/{args.warmup}")
    assert int(status.max().item()) == 0, "a matrix was reported degenerate"

    # events only around the Björck launches, which the rates and the
    # roofline need (each timed launch costs a few microseconds of stream
    # time, which would otherwise inflate the small workloads' step)
    orth.orth_timing_filter("bjorck_", *(("power_",) if args.prescale == "spectral" else ()))
    orth.orth_timing_enable(True)
    orth.orth_timing_reset()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    log(f"[bench] timed {args.steps} steps")
    names = orth.orth_timing_names()
    ktimes = {n: orth.orth_timing_read(n) for n in names}
    # wall time covered by the Björck launches (the small-matrix kernels run
    # on side streams, beside the tiled ones)
    t_bjorck_ms = orth.orth_timing_span("bjorck_")[0] / args.steps
    orth.orth_timing_enable(False)
    orth.orth_timing_filter()

    ms_per_step = (t1 - t0) * 1e3 / args.steps
    value = w.n_layers / (ms_per_step / 1e3)
    shapes = w.matrix_shapes()
    bjorck_flops = wl.algorithmic_bjorck_flops(shapes, w.iters)
    peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS
    bjorck_tflops = bjorck_flops / (t_bjorck_ms / 1e3) / 1e12 if t_bjorck_ms > 0 else None
    step_tflops = bjorck_flops / (ms_per_step / 1e3) / 1e12
    # executed flops of the tiled launches (upper-triangle Gram tiles) plus
    # the small matrices' dense count
    small_flops = wl.algorithmic_bjorck_flops([s_ for s_ in shapes if min(s_) <= 64 and max(s_) <= 128], w.iters)
    tiled_exec = sum(executed_flops(w, n) for n in ("bjorck_bf16_128", "bjorck_bf16_256")) if w.dtype == "bf16" \
        else executed_flops(w, "")
    bjorck_exec_tflops = (tiled_exec + small_flops) / (t_bjorck_ms / 1e3) / 1e12 if t_bjorck_ms > 0 else None

    # roofline of the dominant kernel: algorithmic flops of its launches in
    # the timed region over its measured time (= per-launch average / average
    # launch duration)
    tiled = [n for n in names if n.startswith("bjorck_bf16") or n in ("bjorck_gram_f32", "bjorck_update_f32")]
    roof = None
    if tiled:
        # the fp32 path times its Gram and update launches separately, with
        # equal flops and times within a few percent of each other: report
        # the update launches, which carry the iterate's HBM traffic
        dom = "bjorck_update_f32" if "bjorck_update_f32" in tiled else max(tiled, key=lambda n: ktimes[n][0])
        tot_ms, launches = ktimes[dom]
        if dom.startswith("bjorck_bf16"):
            flops = class_flops(w, dom) * args.steps
        else:   # fp32 path: Gram and update launches are timed separately, each half of the flops
            flops = class_flops(w, "") * args.steps / 2
        achieved = flops / (tot_ms / 1e3) / 1e12
        roof = {"bound": "mfma", "kernel": dom, "achieved": round(achieved, 1), "peak": peak, "unit": "TFLOP/s",
                "frac": round(achieved / peak, 4), "traffic": measured_traffic(dom, w.name),
                "avg_launch_ms": round(tot_ms / launches, 4),
                "algorithmic_flops_per_launch": int(flops / launches)}
        if dom.startswith("bjorck_bf16"):
            # what the MFMA pipes execute: the Gram launches skip the lower
            # tiles of the symmetric E, so the executed rate is below the
            # algorithmic one
            ex = executed_flops(w, dom) * args.steps
            ex_ach = ex / (tot_ms / 1e3) / 1e12
            roof["executed"] = {"achieved": round(ex_ach, 1), "frac": round(ex_ach / peak, 4),
                                "flops_per_launch": int(ex / launches),
                                "note": "upper-triangle Gram tiles plus full update tiles, padded tile grid"}

    power = None
    if args.prescale == "spectral" and "power_dot" in ktimes:
        # HBM roofline of the power-iteration products: each reads every
        # tiled matrix once (the fused small kernel does its own in LDS)
        esz = 2 if w.dtype == "bf16" else 4
        mbytes = sum(r * c * esz for r, c in shapes if not (min(r, c) <= 64 and max(r, c) <= 128))
        tot_ms, launches = ktimes["power_dot"]
        per_launch = mbytes
        ach = per_launch * launches / (tot_ms / 1e3) / 1e9
        power = {"power_iters": args.power_iters,
                 "ms_per_step": round(sum(ktimes[n][0] for n in names if n.startswith("power_")) / args.steps, 4),
                 "roofline": {"bound": "hbm", "kernel": "power_dot", "achieved": round(ach, 1),
                              "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBS, 4),
                              "traffic": None, "avg_launch_ms": round(tot_ms / launches, 4),
                              "algorithmic_bytes_per_launch": per_launch}}

    capply = None
    if args.conv_apply:
        capply = run_conv_apply(w, layers, args.apply_batch, 3, torch, orth, dev)

    expo_rec = None
    if args.expo:
        expo_rec = run_expo(w, ins, 3, torch, orth, dev)

    vjp = None
    if args.vjp:
        vjp = run_vjp(w, ins, outs, layers, status, compute, args.vjp_steps, 1, torch, orth, dev)

    cpu = None
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle sample")
        cpu = cpu_baseline(w)
        if vjp is not None:
            log("[bench] timing the CPU oracle VJP sample")
            vjp["cpu_baseline"] = vjp_cpu_baseline(w)

    if args.copy_calibration:
        # a plain streaming kernel of known traffic: reads 1 GiB, writes 1 GiB
        a = torch.ones(2**28, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        torch.neg(a, out=b)
        torch.cuda.synchronize()

    rec = {
        "metric": METRIC, "value": round(value, 3), "unit": "layers/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic (seeded N(0,1/fan_in) parameters)",
        "config": {"workload": w.name, "matrices": len(shapes), "layers": w.n_layers, "iters": w.iters,
                   "compute": "bf16 operands, fp32 accumulate" if w.dtype == "bf16" else "fp32",
                   "prescale": args.prescale},
        "bjorck_tflops_algorithmic": round(bjorck_tflops, 1) if bjorck_tflops else None,
        "bjorck_pct_peak": round(100 * bjorck_tflops / peak, 2) if bjorck_tflops else None,
        "bjorck_tflops_executed": round(bjorck_exec_tflops, 1) if bjorck_exec_tflops else None,
        "bjorck_pct_peak_executed": round(100 * bjorck_exec_tflops / peak, 2) if bjorck_exec_tflops else None,
        "t_bjorck_ms": round(t_bjorck_ms, 3),
        "step_tflops_algorithmic": round(step_tflops, 1),
        "kernel_ms_per_step": {n: round(ktimes[n][0] / args.steps, 4) for n in names},
        "roofline": roof, "cpu_baseline": cpu,
    }
    if power is not None:
        rec["power_iteration"] = power
    if capply is not None:
        rec["conv_apply"] = capply
    if expo_rec is not None:
        rec["exponentials"] = expo_rec
    if vjp is not None:
        rec["vjp"] = vjp
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
