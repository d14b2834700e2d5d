"""The library's host code (argument validation, planning, workspace layout,
descriptor uploads, plan cache) built for the CPU with AddressSanitizer and
UndefinedBehaviorSanitizer, its HIP runtime calls and kernel launches
replaced by checking stand-ins (tests/host_stub/stub_hip.cpp), and driven
through every batched entry point for all five workloads, their spectral
and saving variants and the error paths (tests/host_stub/driver.cpp), from
one thread and from four at once (then also under ThreadSanitizer).

The stand-ins check that every copy lands in the call's device buffers and
that every table a launch reads lies in the workspace and was uploaded by
the same call; the sanitizers check the host code's own memory accesses
and arithmetic.  No GPU is needed."""

import hashlib
import os
import subprocess

import pytest

from paper_2601_13776_amd import workloads as wl

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
STUB = os.path.join(HERE, "host_stub")
CSRC = os.path.join(ROOT, "paper_2601_13776_amd", "csrc")
BUILD = os.path.join(STUB, "_build")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CLANG = "/opt/rocm/llvm/bin/clang++"
SOURCES = [os.path.join(CSRC, f) for f in ("host.hip", "internal.h", "tile_order.h")] + \
    [os.path.join(ROOT, "include", "orth.h"), os.path.join(STUB, "stub_hip.cpp"), os.path.join(STUB, "driver.cpp")]

# host-side sanitizer flags (each -fsanitize= after -Xarch_host: host code only)
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=undefined"]


# ThreadSanitizer instead (it cannot be combined with AddressSanitizer); its
# application address ranges hold a 1 TiB stand-in device space, not 32 TiB
TSAN = ["-Xarch_host", "-fsanitize=thread", "-DSTUB_ARENA_BITS=40"]


def build_driver(thread=False, planted=False):
    """Compile (once per source state) the sanitized host code, the stand-ins
    and the driver; returns the driver's path.  thread: built with
    ThreadSanitizer instead of AddressSanitizer and UndefinedBehaviorSanitizer;
    planted: with a data race planted in the stand-ins."""
    h = hashlib.sha256()
    for f in SOURCES:
        h.update(open(f, "rb").read())
    tag = h.hexdigest()[:16] + ("_tsan" if thread else "") + ("_race" if planted else "")
    exe = os.path.join(BUILD, f"driver_{tag}")
    if os.path.exists(exe):
        return exe
    os.makedirs(BUILD, exist_ok=True)
    hip = [HIPCC, "-x", "hip", "--offload-host-only", "-O1", "-g", "-std=c++17", "-fPIC", *(TSAN if thread else SAN),
           *(["-DPLANT_RACE"] if planted else []), "-Wno-unused-command-line-argument"]
    host_san = ["-fsanitize=thread"] if thread else ["-fsanitize=address", "-fsanitize=undefined",
                                                     "-fno-sanitize-recover=undefined"]
    objs = []
    procs = []
    for src, obj in ((os.path.join(CSRC, "host.hip"), "host.o"), (os.path.join(STUB, "stub_hip.cpp"), "stub.o")):
        out = os.path.join(BUILD, f"{tag}_{obj}")
        procs.append(subprocess.Popen(hip + ["-c", src, "-o", out], stdout=subprocess.PIPE, stderr=subprocess.STDOUT))
        objs.append(out)
    drv = os.path.join(BUILD, f"{tag}_driver.o")
    procs.append(subprocess.Popen([CLANG, "-O1", "-g", "-std=c++17", *host_san, "-c", os.path.join(STUB, "driver.cpp"),
                                   "-o", drv], stdout=subprocess.PIPE, stderr=subprocess.STDOUT))
    objs.append(drv)
    for p in procs:
        out, _ = p.communicate()
        assert p.returncode == 0, out.decode()[-3000:]
    r = subprocess.run([CLANG, *host_san[:2 if not thread else 1], *objs, "-o", exe + ".tmp", "-lpthread"],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    os.replace(exe + ".tmp", exe)
    return exe


def workload_spec():
    """Driver commands: every workload through the forward, saving forward,
    vector-Jacobian products (recomputing and saved), spectral pre-scaling,
    and the compositions; then error paths with their expected statuses."""
    lines = []
    for name in wl.WORKLOAD_ORDER:
        w = wl.WORKLOADS[name]
        shapes = w.matrix_shapes()
        comp = 1 if w.dtype == "bf16" else 0
        mats = f"{len(shapes)} " + " ".join(f"{r} {c}" for r, c in shapes)
        lines.append(f"# {name}")
        lines.append(f"ortho {w.iters} {comp} {comp} 1 1 0 0 {mats}")
        lines.append(f"ortho {w.iters} {comp} {comp} 2 3 0 0 {mats}")
        if name != "stress_4096x64_32x4096":   # the VJP workspaces scale with T; the forward covers the batch
            for pres, q in ((1, 1), (2, 2)):
                lines.append(f"save 3 {comp} {comp} {pres} {q} 0 0 {mats}")
                lines.append(f"vjp 3 {comp} {comp} {pres} {q} 0 0 0 {mats}")
                lines.append(f"vjp 3 {comp} {comp} {pres} {q} 0 1 0 {mats}")
        convs = [L for L in w.layers if isinstance(L, wl.ConvLayer)]
        if convs:
            geo = f"{len(convs)} " + " ".join(f"{L.cin} {L.cout} {L.k} {L.stride} {L.dilation} {L.groups}"
                                               for L in convs)
            for dt in (0, 1):
                lines.append(f"conv {dt} 0 {geo}")
                lines.append(f"convvjp {dt} 0 {geo}")
                lines.append(f"convsave {dt} 0 {geo}")
    lines.append("# ragged and forced tile sizes")
    lines.append("ortho 4 1 1 1 1 256 0 4 1100 1030 1030 1100 33 17 2048 1000")
    lines.append("ortho 4 1 1 1 1 128 0 3 4096 4096 300 700 1 1")
    lines.append("vjp 4 1 1 2 16 256 0 0 3 1100 1030 64 32 17 33")
    lines.append("# error paths")
    lines.append("ortho 4 0 0 1 1 0 1 2 0 4 8 8")            # rows 0
    lines.append("ortho 4 0 0 1 1 64 1 1 8 8")               # tile 64
    lines.append("ortho 4 0 0 7 1 0 1 1 8 8")                # unknown prescale
    lines.append("ortho 4 0 0 2 0 0 1 1 8 8")                # spectral, no power step
    lines.append("vjp 4 0 0 2 17 0 0 2 1 8 8")               # spectral VJP, 17 power steps
    lines.append("save 4 0 0 2 17 0 2 1 8 8")
    lines.append("conv 0 2 1 4 4 1 2 1 1")                   # k < s
    lines.append("conv 0 2 1 8 8 3 2 2 1")                   # gcd(s, d) != 1
    lines.append("conv 0 1 1 6 8 3 1 1 4")                   # groups do not divide
    lines.append("convvjp 0 2 1 4 4 1 2 1 1")
    return "\n".join(lines) + "\n"


@pytest.mark.slow
def test_host_code_under_sanitizers():
    exe = build_driver()
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], input=workload_spec(), capture_output=True, text=True, env=env, timeout=900)
    tail = (r.stdout[-3000:] + "\n" + r.stderr[-6000:])
    assert r.returncode == 0, tail
    assert "failures 0" in r.stdout, tail
    n_cmds = sum(1 for l in workload_spec().splitlines() if l and not l.startswith("#"))
    assert r.stdout.count("\nok ") + r.stdout.startswith("ok ") == n_cmds, tail


@pytest.mark.slow
@pytest.mark.parametrize("thread", [False, True], ids=["asan-ubsan", "tsan"])
def test_host_code_from_four_threads(thread):
    """Every command of the workload spec from four threads at once, each on
    buffers of its own: the shared plan cache (evicting under concurrent
    users), the staging pool, the per-thread side streams and last errors;
    AddressSanitizer sees a plan or buffer freed under a user, and
    ThreadSanitizer any data race."""
    exe = build_driver(thread=thread)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1", TSAN_OPTIONS="halt_on_error=1")
    r = subprocess.run([exe, "4"], input=workload_spec(), capture_output=True, text=True, env=env, timeout=900)
    tail = (r.stdout[-3000:] + "\n" + r.stderr[-6000:])
    assert r.returncode == 0, tail
    n_cmds = sum(1 for l in workload_spec().splitlines() if l and not l.startswith("#"))
    assert f"threads 4 commands {4 * n_cmds} failures 0" in r.stdout, tail
    assert "WARNING: ThreadSanitizer" not in r.stderr, tail


@pytest.mark.slow
def test_thread_sanitizer_catches_a_planted_race():
    exe = build_driver(thread=True, planted=True)
    r = subprocess.run([exe, "4"], input=workload_spec(), capture_output=True, text=True, timeout=900,
                       env=dict(os.environ, TSAN_OPTIONS="halt_on_error=1"))
    assert r.returncode != 0 and "WARNING: ThreadSanitizer: data race" in r.stderr, r.stderr[-2000:]


@pytest.mark.slow
@pytest.mark.parametrize("which,message", [(0, "table not uploaded by this call"),
                                           (1, "copy destination outside device memory")])
def test_stub_checks_catch_planted_violations(which, message):
    """The stand-ins' own checks: a table read that no copy wrote, and a copy
    past the end of a device buffer, each abort the driver."""
    exe = build_driver()
    r = subprocess.run([exe], input=f"selftest {which}\n", capture_output=True, text=True, timeout=120,
                       env=dict(os.environ, ASAN_OPTIONS="detect_leaks=0"))
    assert r.returncode != 0
    assert "STUB VIOLATION: " + message in r.stderr, r.stderr[-2000:]


def build_tile_order_check(planted=False):
    """The exact-cover checks of the work-list orders (tile_order.h), built
    for the CPU with the same sanitizers (once per source state); planted:
    with a duplicated tile that the checks must catch."""
    srcs = [os.path.join(CSRC, f) for f in ("tile_order.h", "internal.h")] + \
        [os.path.join(ROOT, "include", "orth.h"), os.path.join(STUB, "tile_order_check.cpp")]
    h = hashlib.sha256()
    for f in srcs:
        h.update(open(f, "rb").read())
    exe = os.path.join(BUILD, f"tile_order_check_{'planted_' if planted else ''}{h.hexdigest()[:16]}")
    if os.path.exists(exe):
        return exe
    os.makedirs(BUILD, exist_ok=True)
    r = subprocess.run([HIPCC, "-x", "hip", "--offload-host-only", "-O1", "-g", "-std=c++17", *SAN,
                        *(["-DPLANT_MISTAKE"] if planted else []), "-Wno-unused-command-line-argument",
                        os.path.join(STUB, "tile_order_check.cpp"), "-o", exe + ".tmp"],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    os.replace(exe + ".tmp", exe)
    return exe


@pytest.mark.slow
def test_work_lists_cover_every_tile_once():
    """Gram lists hold every upper tile of every matrix once, update lists
    every tile once, and the XCD reordering is a permutation: the batch
    shapes of the stress and ImageNet-like workloads, edge cases and 150
    random batches."""
    exe = build_tile_order_check()
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300,
                       env=dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1"))
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert "failures 0" in r.stdout and "FAIL" not in r.stdout


@pytest.mark.slow
def test_work_list_checks_catch_a_duplicated_tile():
    exe = build_tile_order_check(planted=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300,
                       env=dict(os.environ, ASAN_OPTIONS="detect_leaks=0"))
    assert r.returncode != 0 and "FAIL" in r.stdout and "Gram tile missing or repeated" in r.stdout

