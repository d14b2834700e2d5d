"""C-ABI checks that need no GPU: the library loads, exports every entry
point the header declares, and its host-side validation and planning agree
with the oracle's geometry rules.  No compute call is made here."""

import ctypes
import os
import re

import pytest

from oracle import aoc
from paper_2601_13776_amd import orth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "orth.h")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(orth._LIB_PATH):
        from paper_2601_13776_amd import build
        build.build(verbose=False)
    return orth.lib()


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(orth_\w+)\s*\(", text, flags=re.M))


def test_header_symbols_exported(L):
    names = header_functions()
    assert len(names) >= 15
    for name in names:
        assert hasattr(L, name), f"{name} declared in orth.h but not exported"
    assert names == set(orth.EXPORTED)


def test_status_strings(L):
    assert L.orth_status_string(0) == b"ok"
    assert b"workspace" in L.orth_status_string(3)
    assert L.orth_version() >= 100


GEOMS = [(16, 16, 3, 1, 1, 1), (64, 128, 3, 2, 1, 1), (128, 512, 2, 2, 1, 1), (256, 256, 3, 1, 1, 4),
         (256, 256, 3, 1, 2, 1), (8, 8, 1, 1, 1, 1), (6, 6, 5, 2, 3, 3), (4, 4, 1, 2, 1, 1),
         (4, 4, 3, 2, 2, 1), (4, 4, 3, 1, 1, 3), (0, 4, 3, 1, 1, 1), (2, 4, 3, 1, 1, 2), (4, 4, 3, 1, 0, 1),
         (3, 64, 3, 1, 1, 1), (64, 3, 3, 1, 1, 1), (64, 64, 7, 1, 1, 1), (32, 64, 4, 2, 1, 1), (48, 48, 3, 1, 2, 3),
         (16, 32, 2, 2, 1, 2), (12, 12, 5, 1, 2, 2), (16, 16, 3, 1, 1, 16), (8, 8, 3, 2, 1, 8)]


@pytest.mark.parametrize("geom", GEOMS)
def test_param_shapes_agree_with_oracle(L, geom):
    try:
        want = aoc.param_shapes(*geom)
        kind = None
    except aoc.GeometryError as e:
        want, kind = None, e.kind
    g = orth.orth_conv_geom(*geom)
    out = [ctypes.c_int32() for _ in range(5)]
    rc = L.orth_aoc_param_shapes(ctypes.byref(g), *[ctypes.byref(o) for o in out])
    if kind is None:
        assert rc == orth.ORTH_OK
        assert tuple(o.value for o in out) == want
    else:
        assert rc == {"invalid": orth.ORTH_EINVAL, "unsupported": orth.ORTH_EUNSUPPORTED}[kind]
        assert L.orth_last_error()


def _mats(shapes, base=0x10000):
    arr = (orth.orth_mat * len(shapes))()
    for i, (r, c) in enumerate(shapes):
        arr[i] = orth.orth_mat(base + 0x100000 * i, base + 0x100000 * i + 0x80000, r, c, c, c)
    return arr


def _ws_size(L, shapes, **kw):
    opts = orth.orth_bjorck_opts(kw.get("iters", 5), kw.get("beta", 0.5), 1, kw.get("dt", 0), kw.get("dt", 0),
                                 kw.get("compute", 0), 1, None, kw.get("tile", 0))
    n = ctypes.c_size_t()
    rc = L.orth_orthogonalize_workspace_size(_mats(shapes), len(shapes), ctypes.byref(opts), ctypes.byref(n))
    return rc, n.value


def test_workspace_sizes(L):
    rc, small = _ws_size(L, [(16, 16), (16, 8), (8, 16)])
    assert rc == 0 and 0 < small < 1 << 16        # tables only
    rc, big = _ws_size(L, [(4096, 4096)], compute=1, dt=1)
    # fp32 iterate + two bf16 copies (ping-pong) + bf16 E
    assert rc == 0 and 4096 * 4096 * (4 + 2 + 2 + 2) <= big < 4096 * 4096 * 11
    # fp32 products, output not laid out as the iterate: two fp32 iterates
    # (ping-pong) + the transposed iterate + E
    f32 = _ws_out(L, [(512, 256)], 0, 0, 0, ld_pad=4)
    assert f32 >= 512 * 256 * (4 + 4 + 4) + 256 * 256 * 4


def _ws_out(L, shapes, compute, in_dt, out_dt, iters=5, ld_pad=0, out_off=0, inplace=False):
    arr = (orth.orth_mat * len(shapes))()
    for i, (r, c) in enumerate(shapes):
        src = 0x10000 + 0x4000000 * i
        dst = src if inplace else src + 0x2000000 + out_off
        arr[i] = orth.orth_mat(src, dst, r, c, c + (ld_pad if inplace else 0), c + ld_pad)
    opts = orth.orth_bjorck_opts(iters, 0.5, 1, in_dt, out_dt, compute, 1, None, 0)
    n = ctypes.c_size_t()
    assert L.orth_orthogonalize_workspace_size(arr, len(shapes), ctypes.byref(opts), ctypes.byref(n)) == 0
    return n.value


def test_output_holds_iterate(L):
    """An fp32 output laid out as the fp32 iterate (tall, no padding,
    ld_out == cols, 16-byte aligned) serves as the buffer the last step
    writes: exactly one fp32 iterate less workspace; any other output keeps
    the workspace buffer (and the write-out pass)."""
    sq = [(4096, 4096)]
    full = _ws_out(L, sq, 1, 1, 0, ld_pad=8)
    assert full - _ws_out(L, sq, 1, 1, 0) == 4096 * 4096 * 4
    assert _ws_out(L, sq, 1, 1, 0, out_off=8) == full           # misaligned output
    assert _ws_out(L, sq, 1, 1, 1) == full                      # bf16 output
    assert _ws_out(L, [(4096, 8192)], 1, 1, 0) == _ws_out(L, [(4096, 8192)], 1, 1, 0, ld_pad=8)   # wide
    assert _ws_out(L, [(1000, 1000)], 1, 1, 0) == _ws_out(L, [(1000, 1000)], 1, 1, 0, ld_pad=8)   # padded
    assert _ws_out(L, [(100, 40)], 0, 0, 0) == _ws_out(L, [(100, 40)], 0, 0, 0, ld_pad=8)         # fused kernel
    for iters in (0, 5, 6):   # fp32 products: X_T in slot T mod 2, either slot
        full = _ws_out(L, [(512, 256)], 0, 0, 0, iters=iters, ld_pad=4)
        assert full - _ws_out(L, [(512, 256)], 0, 0, 0, iters=iters) == 512 * 256 * 4
        assert full - _ws_out(L, [(512, 256)], 0, 0, 0, iters=iters, inplace=True) == 512 * 256 * 4
        assert _ws_out(L, [(512, 256)], 0, 0, 0, iters=iters, ld_pad=4, inplace=True) == full


@pytest.mark.parametrize("kw,shapes,code", [
    (dict(beta=0.75), [(4, 4)], orth.ORTH_EINVAL),
    (dict(beta=0.0), [(4, 4)], orth.ORTH_EINVAL),
    (dict(iters=-1), [(4, 4)], orth.ORTH_EINVAL),
    (dict(compute=7), [(4, 4)], orth.ORTH_EINVAL),
    (dict(dt=3), [(4, 4)], orth.ORTH_EINVAL),
    (dict(), [(0, 4)], orth.ORTH_EINVAL),
    (dict(), [(4, 0)], orth.ORTH_EINVAL),
    (dict(tile=64), [(4, 4)], orth.ORTH_EINVAL),
    (dict(tile=512, compute=1), [(4, 4)], orth.ORTH_EINVAL),
])
def test_invalid_orthogonalize_args(L, kw, shapes, code):
    rc, _ = _ws_size(L, shapes, **kw)
    assert rc == code
    opts = orth.orth_bjorck_opts(kw.get("iters", 5), kw.get("beta", 0.5), 1, kw.get("dt", 0), kw.get("dt", 0),
                                 kw.get("compute", 0), 1, None, kw.get("tile", 0))
    rc = L.orth_orthogonalize_batched(_mats(shapes), len(shapes), ctypes.byref(opts), None, 0, None, None)
    assert rc == code


def test_tile_class_choice(L):
    """bf16 matrices with min(rows, cols) >= 1024 are padded to the chosen
    tile edge: a lone 1100 x 1030 matrix gets 128-tiles by occupancy (its
    20 tiles of 256 would leave most compute units idle), 256-tiles when
    forced; a batch with >= 1024 tiles of 256 gets 256-tiles."""
    one = [(1100, 1030)]
    _, auto = _ws_size(L, one, compute=1, dt=1)
    _, t128 = _ws_size(L, one, compute=1, dt=1, tile=128)
    _, t256 = _ws_size(L, one, compute=1, dt=1, tile=256)
    assert auto == t128 < t256
    many = [(4096, 4096)] * 4                        # 4 x 256 tiles of 256
    _, auto = _ws_size(L, many, compute=1, dt=1)
    _, t256 = _ws_size(L, many, compute=1, dt=1, tile=256)
    assert auto == t256
    # fp32 products ignore the option
    _, a = _ws_size(L, one)
    _, b = _ws_size(L, one, tile=256)
    assert a == b


def test_bad_leading_dim_and_inplace(L):
    arr = (orth.orth_mat * 1)()
    arr[0] = orth.orth_mat(0x1000, 0x2000, 8, 8, 4, 8)
    opts = orth.orth_bjorck_opts(3, 0.5, 1, 0, 0, 0)
    n = ctypes.c_size_t()
    assert L.orth_orthogonalize_workspace_size(arr, 1, ctypes.byref(opts), ctypes.byref(n)) == orth.ORTH_EINVAL
    arr[0] = orth.orth_mat(0x1000, 0x1000, 8, 8, 8, 8)
    opts = orth.orth_bjorck_opts(3, 0.5, 1, 1, 0, 0)          # bf16 in, fp32 out, in place
    assert L.orth_orthogonalize_workspace_size(arr, 1, ctypes.byref(opts), ctypes.byref(n)) == orth.ORTH_EINVAL


def test_workspace_errors_before_launch(L):
    opts = orth.orth_bjorck_opts(3, 0.5, 1, 0, 0, 0)
    shapes = [(256, 128)]
    rc, need = _ws_size(L, shapes)
    assert rc == 0
    assert L.orth_orthogonalize_batched(_mats(shapes), 1, ctypes.byref(opts), None, need, None, None) \
        == orth.ORTH_EWORKSPACE
    assert L.orth_orthogonalize_batched(_mats(shapes), 1, ctypes.byref(opts), 0x100000, need - 1, None, None) \
        == orth.ORTH_EWORKSPACE
    assert L.orth_orthogonalize_batched(_mats(shapes), 1, ctypes.byref(opts), 0x100010, need, None, None) \
        == orth.ORTH_EWORKSPACE
    assert b"aligned" in L.orth_last_error()
    # an empty batch is a no-op
    assert L.orth_orthogonalize_batched(None, 0, ctypes.byref(opts), None, 0, None, None) == orth.ORTH_OK


def test_noalloc_errors_before_the_device(L):
    """The allocation-free entry point validates like the workspace one and
    rejects a batch larger than its fixed scratch with ORTH_EWORKSPACE, all
    on the host (no GPU here)."""
    opts = orth.orth_bjorck_opts(3, 0.5, 1, 0, 0, 0)
    assert L.orth_orthogonalize_batched_noalloc(None, 0, ctypes.byref(opts), None, None) == orth.ORTH_OK
    assert L.orth_orthogonalize_batched_noalloc(_mats([(0, 4)]), 1, ctypes.byref(opts), None, None) \
        == orth.ORTH_EINVAL
    bad = orth.orth_bjorck_opts(3, 0.75, 1, 0, 0, 0)
    assert L.orth_orthogonalize_batched_noalloc(_mats([(8, 4)]), 1, ctypes.byref(bad), None, None) \
        == orth.ORTH_EINVAL
    big = [(4096, 2048)]
    rc, need = _ws_size(L, big)
    assert rc == 0 and need > orth.ORTH_NOALLOC_SCRATCH_BYTES
    assert L.orth_orthogonalize_batched_noalloc(_mats(big), 1, ctypes.byref(opts), None, None) \
        == orth.ORTH_EWORKSPACE
    assert b"holds 67108864" in L.orth_last_error()


def test_conv_validation(L):
    d = (orth.orth_conv_desc * 1)()
    d[0] = orth.orth_conv_desc(orth.orth_conv_geom(4, 4, 3, 2, 2, 1), 0x1000, 0x2000, 0x3000)
    n = ctypes.c_size_t()
    assert L.orth_build_conv_kernels_workspace_size(d, 1, 0, ctypes.byref(n)) == orth.ORTH_EUNSUPPORTED
    d[0] = orth.orth_conv_desc(orth.orth_conv_geom(16, 16, 3, 1, 1, 1), 0x1000, None, 0x3000)
    assert L.orth_build_conv_kernels_workspace_size(d, 1, 0, ctypes.byref(n)) == orth.ORTH_EINVAL
    d[0] = orth.orth_conv_desc(orth.orth_conv_geom(16, 16, 3, 1, 1, 1), 0x1000, 0x2000, 0x3000)
    assert L.orth_build_conv_kernels_workspace_size(d, 1, 0, ctypes.byref(n)) == orth.ORTH_OK
    # two tap buffers + products (9 taps of 16x16) + 4 projectors 16x16, fp32
    assert n.value >= (3 * 9 * 256 + 4 * 256) * 4
    d[0] = orth.orth_conv_desc(orth.orth_conv_geom(128, 512, 2, 2, 1, 1), 0x1000, None, 0x3000)
    assert L.orth_build_conv_kernels_workspace_size(d, 1, 0, ctypes.byref(n)) == orth.ORTH_OK


def test_check_validation(L):
    a = orth.orth_check_args()
    a.mode = 9
    n = ctypes.c_size_t()
    assert L.orth_check_workspace_size(ctypes.byref(a), ctypes.byref(n)) == orth.ORTH_EINVAL
    a.mode = orth.ORTH_CHECK_CONV
    a.geom = orth.orth_conv_geom(16, 16, 3, 2, 1, 1)
    a.kernel, a.x, a.kernel_dtype = 0x1000, 0x2000, 0
    a.batch, a.height, a.width = 2, 15, 16
    assert L.orth_check_workspace_size(ctypes.byref(a), ctypes.byref(n)) == orth.ORTH_EINVAL  # 15 % 2
    a.height = 16
    assert L.orth_check_workspace_size(ctypes.byref(a), ctypes.byref(n)) == orth.ORTH_OK


def _vjp_mats(shapes, alias=None):
    arr = (orth.orth_vjp_mat * len(shapes))()
    for i, (r, c) in enumerate(shapes):
        w = 0x10000 + 0x1000000 * i
        go = w + 0x400000
        gi = {"grad_out": go, "w": w}.get(alias, w + 0x800000)
        arr[i] = orth.orth_vjp_mat(w, go, gi, r, c, c, c, c)
    return arr


def _vjp_ws(L, shapes, iters=5, compute=0, dt=0, prescale=1, beta=0.5, alias=None, tile=0):
    opts = orth.orth_bjorck_opts(iters, beta, prescale, dt, dt, compute, 1, None, tile)
    n = ctypes.c_size_t()
    rc = L.orth_orthogonalize_vjp_workspace_size(_vjp_mats(shapes, alias), len(shapes), ctypes.byref(opts),
                                                 ctypes.byref(n))
    return rc, n.value


def test_save_workspace_matches_vjp(L):
    """A saving forward fills a vector-Jacobian workspace: its size query
    equals the VJP's for the same shapes and options, in every bucket
    (fused small, fp32 tiles, bf16 tiles of both classes)."""
    shapes = [(16, 8), (100, 70), (300, 200), (2048, 1024), (8, 16)]
    for compute, dt in ((0, 0), (1, 1), (1, 0)):
        for iters in (0, 1, 6):
            opts = orth.orth_bjorck_opts(iters, 0.5, 1, dt, dt, compute, 1, None, 0)
            n = ctypes.c_size_t()
            assert L.orth_orthogonalize_save_workspace_size(_mats(shapes), len(shapes), ctypes.byref(opts),
                                                            ctypes.byref(n)) == orth.ORTH_OK
            rc, v = _vjp_ws(L, shapes, iters=iters, compute=compute, dt=dt)
            assert rc == orth.ORTH_OK and n.value == v, (compute, dt, iters)


def test_save_and_saved_flag_errors(L):
    n = ctypes.c_size_t()
    opts = orth.orth_bjorck_opts(3, 0.5, 1, 0, 0, 0, 1, None, 0, 1)     # saved = 1: not for the forward
    assert L.orth_orthogonalize_save_workspace_size(_mats([(64, 32)]), 1, ctypes.byref(opts),
                                                    ctypes.byref(n)) == orth.ORTH_EINVAL
    opts = orth.orth_bjorck_opts(3, 0.5, 1, 0, 0, 0, 1, None, 0, 2)     # saved must be 0 or 1
    rc, _ = _vjp_ws(L, [(64, 32)])
    assert rc == orth.ORTH_OK
    assert L.orth_orthogonalize_vjp_workspace_size(_vjp_mats([(64, 32)]), 1, ctypes.byref(opts),
                                                   ctypes.byref(n)) == orth.ORTH_EINVAL
    inplace = (orth.orth_mat * 1)()
    inplace[0] = orth.orth_mat(0x10000, 0x10000, 64, 32, 32, 32)
    opts = orth.orth_bjorck_opts(3, 0.5, 1, 0, 0, 0, 1, None, 0)
    assert L.orth_orthogonalize_save_workspace_size(inplace, 1, ctypes.byref(opts), ctypes.byref(n)) \
        == orth.ORTH_EINVAL
    assert L.orth_orthogonalize_save_batched(inplace, 1, ctypes.byref(opts), None, 0, None, None) == orth.ORTH_EINVAL
    spectral = orth.orth_bjorck_opts(3, 0.5, 2, 0, 0, 0, 17, 0x1000, 0)   # over 16 power steps
    assert L.orth_orthogonalize_save_workspace_size(_mats([(64, 32)]), 1, ctypes.byref(spectral),
                                                    ctypes.byref(n)) == orth.ORTH_EUNSUPPORTED
    # too small a workspace: rejected before anything is enqueued
    rc, need = _vjp_ws(L, [(64, 32)], iters=3)
    assert L.orth_orthogonalize_save_batched(_mats([(64, 32)]), 1, ctypes.byref(opts), 0x100000, need - 1, None,
                                             None) == orth.ORTH_EWORKSPACE


def test_conv_save_workspace_matches_vjp(L):
    """A saving composition fills a composition-VJP workspace: its size
    query equals the VJP's for the same geometries and dtype."""
    geoms = [(16, 16, 3, 1, 1, 1), (16, 32, 2, 2, 1, 1), (32, 32, 3, 1, 1, 4), (6, 6, 5, 2, 3, 3), (8, 8, 1, 1, 1, 1)]
    fwd = (orth.orth_conv_desc * len(geoms))()
    vjp = (orth.orth_conv_vjp_desc * len(geoms))()
    for i, g in enumerate(geoms):
        base = 0x100000 * (i + 1)
        has_proj = g[2] > g[3]
        fwd[i] = orth.orth_conv_desc(orth.orth_conv_geom(*g), base, base + 0x10000 if has_proj else None, base + 0x20000)
        vjp[i] = orth.orth_conv_vjp_desc(orth.orth_conv_geom(*g), base, base + 0x10000 if has_proj else None,
                                         base + 0x30000, base + 0x40000, base + 0x50000 if has_proj else None)
    for dt in (0, 1):
        a, b = ctypes.c_size_t(), ctypes.c_size_t()
        assert L.orth_build_conv_kernels_save_workspace_size(fwd, len(geoms), dt, ctypes.byref(a)) == orth.ORTH_OK
        assert L.orth_build_conv_kernels_vjp_workspace_size(vjp, len(geoms), dt, ctypes.byref(b)) == orth.ORTH_OK
        assert a.value == b.value > 0
    bad = (orth.orth_conv_desc * 1)()
    bad[0] = orth.orth_conv_desc(orth.orth_conv_geom(16, 16, 3, 1, 1, 1), 0x1000, None, 0x3000)   # proj missing
    n = ctypes.c_size_t()
    assert L.orth_build_conv_kernels_save_workspace_size(bad, 1, 0, ctypes.byref(n)) == orth.ORTH_EINVAL


def test_vjp_workspace_grows_with_saved_steps(L):
    """The VJP keeps X_t and E_t of every step: fp32 products hold
    T (2 M N + N^2) fp32 values beside a few fixed buffers (X_t also
    transposed, so that every product reads K-contiguous operands), bf16
    products T (M N + N^2) bf16 values."""
    rc, w5 = _vjp_ws(L, [(256, 128)], iters=5)
    rc2, w10 = _vjp_ws(L, [(256, 128)], iters=10)
    assert rc == rc2 == orth.ORTH_OK
    assert w10 - w5 == pytest.approx(5 * (2 * 256 * 128 + 128 * 128) * 4, rel=0.01)
    rc, b5 = _vjp_ws(L, [(2048, 1024)], iters=5, compute=1, dt=1)
    rc2, b10 = _vjp_ws(L, [(2048, 1024)], iters=10, compute=1, dt=1)
    assert rc == rc2 == orth.ORTH_OK
    assert b10 - b5 == pytest.approx(5 * (2048 * 1024 + 1024 * 1024) * 2, rel=0.01)


@pytest.mark.parametrize("kw,code", [
    (dict(iters=-1), orth.ORTH_EINVAL),
    (dict(iters=5000), orth.ORTH_EINVAL),
    (dict(beta=0.7), orth.ORTH_EINVAL),
    (dict(prescale=3), orth.ORTH_EINVAL),
    (dict(compute=2), orth.ORTH_EINVAL),
    (dict(alias="grad_out"), orth.ORTH_OK),
    (dict(alias="w"), orth.ORTH_OK),
    (dict(iters=0), orth.ORTH_OK),
    (dict(tile=100), orth.ORTH_EINVAL),
    (dict(tile=256, compute=1, dt=1), orth.ORTH_OK),
])
def test_vjp_validation(L, kw, code):
    rc, _ = _vjp_ws(L, [(64, 32), (16, 48)], **kw)
    assert rc == code


def test_vjp_rejects_bad_matrices(L):
    opts = orth.orth_bjorck_opts(3, 0.5, 1, 0, 0, 0)
    n = ctypes.c_size_t()
    arr = _vjp_mats([(8, 4)])
    arr[0].grad_in = None
    assert L.orth_orthogonalize_vjp_workspace_size(arr, 1, ctypes.byref(opts), ctypes.byref(n)) == orth.ORTH_EINVAL
    arr = _vjp_mats([(8, 4)])
    arr[0].ld_grad_out = 3
    assert L.orth_orthogonalize_vjp_workspace_size(arr, 1, ctypes.byref(opts), ctypes.byref(n)) == orth.ORTH_EINVAL
    # aliasing grad_out with a different dtype
    opts = orth.orth_bjorck_opts(3, 0.5, 1, 1, 0, 0)
    arr = _vjp_mats([(8, 4)], alias="grad_out")
    assert L.orth_orthogonalize_vjp_workspace_size(arr, 1, ctypes.byref(opts), ctypes.byref(n)) == orth.ORTH_EINVAL
    assert b"alias" in L.orth_last_error()


def test_conv_vjp_validation(L):
    n = ctypes.c_size_t()
    arr = (orth.orth_conv_vjp_desc * 1)()
    arr[0] = orth.orth_conv_vjp_desc(orth.orth_conv_geom(16, 16, 3, 1, 1, 1), 0x1000, 0x2000, 0x3000, 0x4000, 0x5000)
    assert L.orth_build_conv_kernels_vjp_workspace_size(arr, 1, 0, ctypes.byref(n)) == orth.ORTH_OK
    assert n.value > 0
    arr[0].grad_proj = None
    assert L.orth_build_conv_kernels_vjp_workspace_size(arr, 1, 0, ctypes.byref(n)) == orth.ORTH_EINVAL
    # k == s needs no projector gradient
    arr[0] = orth.orth_conv_vjp_desc(orth.orth_conv_geom(16, 32, 2, 2, 1, 1), 0x1000, None, 0x3000, 0x4000, None)
    assert L.orth_build_conv_kernels_vjp_workspace_size(arr, 1, 0, ctypes.byref(n)) == orth.ORTH_OK
    arr[0] = orth.orth_conv_vjp_desc(orth.orth_conv_geom(16, 16, 1, 2, 1, 1), 0x1000, None, 0x3000, 0x4000, None)
    assert L.orth_build_conv_kernels_vjp_workspace_size(arr, 1, 0, ctypes.byref(n)) == orth.ORTH_EUNSUPPORTED


@pytest.mark.parametrize("q,u,code", [(1, 0x1000, orth.ORTH_OK), (0, 0x1000, orth.ORTH_EINVAL),
                                      (1025, 0x1000, orth.ORTH_EINVAL), (2, None, orth.ORTH_EINVAL)])
def test_spectral_validation(L, q, u, code):
    opts = orth.orth_bjorck_opts(5, 0.5, orth.ORTH_PRESCALE_SPECTRAL, 0, 0, 0, q, u)
    n = ctypes.c_size_t()
    rc = L.orth_orthogonalize_workspace_size(_mats([(64, 32), (300, 200)]), 2, ctypes.byref(opts), ctypes.byref(n))
    assert rc == code


def test_vjp_spectral_validation(L):
    """The VJP through spectral pre-scaling takes 1..16 power steps, needs the
    cached vectors unless it reuses a saving forward's workspace, and its
    workspace grows with the number of power steps."""
    n = ctypes.c_size_t()
    mats = _vjp_mats([(64, 32), (300, 200)])

    def size(q, u, saved=0):
        opts = orth.orth_bjorck_opts(5, 0.5, orth.ORTH_PRESCALE_SPECTRAL, 0, 0, 0, q, u, 0, saved)
        rc = L.orth_orthogonalize_vjp_workspace_size(mats, 2, ctypes.byref(opts), ctypes.byref(n))
        return rc, n.value

    rc1, n1 = size(1, 0x1000)
    rc3, n3 = size(3, 0x1000)
    assert rc1 == rc3 == orth.ORTH_OK and n3 > n1
    assert size(17, 0x1000)[0] == orth.ORTH_EUNSUPPORTED
    assert size(0, 0x1000)[0] == orth.ORTH_EINVAL
    assert size(1, None)[0] == orth.ORTH_EINVAL
    assert size(1, None, saved=1) == (orth.ORTH_OK, n1)
    # the saving forward lays out the same workspace
    opts = orth.orth_bjorck_opts(5, 0.5, orth.ORTH_PRESCALE_SPECTRAL, 0, 0, 0, 1, 0x1000)
    arr = (orth.orth_mat * 2)()
    arr[0] = orth.orth_mat(0x1000, 0x2000, 64, 32, 32, 32)
    arr[1] = orth.orth_mat(0x3000, 0x4000, 300, 200, 200, 200)
    assert L.orth_orthogonalize_save_workspace_size(arr, 2, ctypes.byref(opts), ctypes.byref(n)) == orth.ORTH_OK
    assert n.value == n1


@pytest.mark.parametrize("kw,code", [
    (dict(), orth.ORTH_OK), (dict(height=9), orth.ORTH_EINVAL), (dict(batch=0), orth.ORTH_EINVAL),
    (dict(same=True), orth.ORTH_EINVAL), (dict(kernel_dtype=7), orth.ORTH_EINVAL),
    (dict(geom=(4, 4, 1, 2, 1, 1)), orth.ORTH_EUNSUPPORTED),
])
def test_conv_apply_validation(L, kw, code):
    """Only invalid arguments are exercised here (a valid call would launch)."""
    if code == orth.ORTH_OK:
        return
    geom = kw.get("geom", (4, 8, 3, 2, 1, 1))
    a = orth.orth_conv_apply_args(orth.orth_conv_geom(*geom), 0x1000, kw.get("kernel_dtype", 0), 0, 0x2000,
                                  0x2000 if kw.get("same") else 0x3000, kw.get("batch", 2), kw.get("height", 8), 8)
    assert L.orth_conv_apply(ctypes.byref(a), None) == code


@pytest.mark.parametrize("kw,code", [
    (dict(), orth.ORTH_OK), (dict(terms=0), orth.ORTH_EINVAL), (dict(terms=65), orth.ORTH_EINVAL),
    (dict(q=0), orth.ORTH_EINVAL), (dict(u=None), orth.ORTH_EINVAL), (dict(shape=(8, 6)), orth.ORTH_EINVAL),
])
def test_exp_map_validation(L, kw, code):
    shape = kw.get("shape", (64, 64))
    opts = orth.orth_exp_opts(kw.get("terms", 12), kw.get("q", 1), kw.get("u", 0x1000), 0, 0)
    n = ctypes.c_size_t()
    rc = L.orth_exp_map_workspace_size(_mats([shape, (130, 130)]), 2, ctypes.byref(opts), ctypes.byref(n))
    assert rc == code


@pytest.mark.parametrize("kw,code", [
    (dict(), orth.ORTH_OK), (dict(k=4), orth.ORTH_EUNSUPPORTED), (dict(terms=0), orth.ORTH_EINVAL),
    (dict(c=0), orth.ORTH_EINVAL), (dict(scale=float("nan")), orth.ORTH_EINVAL), (dict(same=True), orth.ORTH_EINVAL),
])
def test_conv_exp_validation(L, kw, code):
    d = (orth.orth_conv_exp_desc * 1)()
    d[0] = orth.orth_conv_exp_desc(kw.get("c", 16), kw.get("k", 3), kw.get("terms", 6), kw.get("scale", 1.0), 0x1000,
                                   0x1000 if kw.get("same") else 0x2000)
    n = ctypes.c_size_t()
    assert L.orth_conv_exp_workspace_size(d, 1, 0, ctypes.byref(n)) == code
    if code == orth.ORTH_OK:
        # tables plus L (9 taps), E and two power grids of 13 x 13 taps of 16 x 16 fp32
        assert n.value >= (9 + 3 * 169) * 256 * 4
