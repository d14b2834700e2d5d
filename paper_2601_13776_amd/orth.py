"""Thin ctypes binding of liborth (include/orth.h).

Argument marshalling only: every step of the path runs in the HIP library.
Functions keep the C names.  Tensors are torch tensors on the GPU; the
library runs on torch's current stream.  If liborth.so is missing the first
call raises: there is no fallback implementation.
"""

import ctypes
import os

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "liborth.so")
_lib = None

ORTH_OK, ORTH_EINVAL, ORTH_EUNSUPPORTED, ORTH_EWORKSPACE, ORTH_EHIP = range(5)
ORTH_F32, ORTH_BF16 = 0, 1
ORTH_COMPUTE_F32, ORTH_COMPUTE_BF16 = 0, 1
ORTH_PRESCALE_NONE, ORTH_PRESCALE_FROBENIUS, ORTH_PRESCALE_SPECTRAL = 0, 1, 2
ORTH_CHECK_GRAM, ORTH_CHECK_CONV, ORTH_CHECK_CONV_ADJOINT = 0, 1, 2
ORTH_NOALLOC_SCRATCH_BYTES = 64 << 20   # the allocation-free entry point's device scratch per GPU

EXPORTED = [
    "orth_orthogonalize_workspace_size", "orth_orthogonalize_batched", "orth_orthogonalize_batched_noalloc",
    "orth_orthogonalize_vjp_workspace_size", "orth_orthogonalize_vjp_batched",
    "orth_orthogonalize_save_workspace_size", "orth_orthogonalize_save_batched", "orth_aoc_param_shapes",
    "orth_build_conv_kernels_workspace_size", "orth_build_conv_kernels_batched", "orth_build_conv_kernel",
    "orth_build_conv_kernels_vjp_workspace_size", "orth_build_conv_kernels_vjp_batched",
    "orth_build_conv_kernels_save_workspace_size", "orth_build_conv_kernels_save_batched",
    "orth_build_conv_kernels_vjp_saved_batched", "orth_conv_apply",
    "orth_exp_map_workspace_size", "orth_exp_map_batched", "orth_conv_exp_workspace_size", "orth_conv_exp_batched",
    "orth_check_workspace_size", "orth_check_norm", "orth_status_string", "orth_last_error",
    "orth_version", "orth_timing_enable", "orth_timing_filter", "orth_timing_reset", "orth_timing_read",
    "orth_timing_span", "orth_timing_names",
]


class OrthError(RuntimeError):
    def __init__(self, code, where):
        self.code = code
        msg = lib().orth_last_error().decode()
        super().__init__(f"{where}: {lib().orth_status_string(code).decode()} ({msg})")


class orth_mat(ctypes.Structure):
    _fields_ = [("in_", ctypes.c_void_p), ("out", ctypes.c_void_p), ("rows", ctypes.c_int32),
                ("cols", ctypes.c_int32), ("ld_in", ctypes.c_int64), ("ld_out", ctypes.c_int64)]


class orth_bjorck_opts(ctypes.Structure):
    _fields_ = [("iters", ctypes.c_int32), ("beta", ctypes.c_float), ("prescale", ctypes.c_int32),
                ("in_dtype", ctypes.c_int32), ("out_dtype", ctypes.c_int32), ("compute", ctypes.c_int32),
                ("power_iters", ctypes.c_int32), ("u", ctypes.c_void_p), ("tile", ctypes.c_int32),
                ("saved", ctypes.c_int32)]


class orth_vjp_mat(ctypes.Structure):
    _fields_ = [("w", ctypes.c_void_p), ("grad_out", ctypes.c_void_p), ("grad_in", ctypes.c_void_p),
                ("rows", ctypes.c_int32), ("cols", ctypes.c_int32), ("ld_w", ctypes.c_int64),
                ("ld_grad_out", ctypes.c_int64), ("ld_grad_in", ctypes.c_int64)]


class orth_exp_opts(ctypes.Structure):
    _fields_ = [("terms", ctypes.c_int32), ("power_iters", ctypes.c_int32), ("u", ctypes.c_void_p),
                ("in_dtype", ctypes.c_int32), ("out_dtype", ctypes.c_int32)]


class orth_conv_exp_desc(ctypes.Structure):
    _fields_ = [("channels", ctypes.c_int32), ("k", ctypes.c_int32), ("terms", ctypes.c_int32),
                ("scale", ctypes.c_float), ("kernel", ctypes.c_void_p), ("out", ctypes.c_void_p)]


class orth_conv_geom(ctypes.Structure):
    _fields_ = [("cin", ctypes.c_int32), ("cout", ctypes.c_int32), ("k", ctypes.c_int32),
                ("stride", ctypes.c_int32), ("dilation", ctypes.c_int32), ("groups", ctypes.c_int32)]


class orth_conv_desc(ctypes.Structure):
    _fields_ = [("geom", orth_conv_geom), ("rko", ctypes.c_void_p), ("proj", ctypes.c_void_p),
                ("kernel", ctypes.c_void_p)]


class orth_conv_vjp_desc(ctypes.Structure):
    _fields_ = [("geom", orth_conv_geom), ("rko", ctypes.c_void_p), ("proj", ctypes.c_void_p),
                ("grad_kernel", ctypes.c_void_p), ("grad_rko", ctypes.c_void_p), ("grad_proj", ctypes.c_void_p)]


class orth_conv_apply_args(ctypes.Structure):
    _fields_ = [("geom", orth_conv_geom), ("kernel", ctypes.c_void_p), ("kernel_dtype", ctypes.c_int32),
                ("transposed", ctypes.c_int32), ("x", ctypes.c_void_p), ("y", ctypes.c_void_p),
                ("batch", ctypes.c_int32), ("height", ctypes.c_int32), ("width", ctypes.c_int32)]


class orth_check_args(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int32), ("mats", ctypes.POINTER(orth_mat)), ("n_mats", ctypes.c_int32),
                ("mat_dtype", ctypes.c_int32), ("kernel", ctypes.c_void_p), ("kernel_dtype", ctypes.c_int32),
                ("geom", orth_conv_geom), ("x", ctypes.c_void_p), ("batch", ctypes.c_int32),
                ("height", ctypes.c_int32), ("width", ctypes.c_int32)]


def lib():
    """Load liborth.so (once)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is missing: build it with `python -m paper_2601_13776_amd.build`")
        L = ctypes.CDLL(_LIB_PATH)
        vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        P = ctypes.POINTER
        L.orth_orthogonalize_workspace_size.argtypes = [P(orth_mat), i32, P(orth_bjorck_opts), P(sz)]
        L.orth_orthogonalize_batched.argtypes = [P(orth_mat), i32, P(orth_bjorck_opts), vp, sz, vp, vp]
        L.orth_orthogonalize_batched_noalloc.argtypes = [P(orth_mat), i32, P(orth_bjorck_opts), vp, vp]
        L.orth_orthogonalize_vjp_workspace_size.argtypes = [P(orth_vjp_mat), i32, P(orth_bjorck_opts), P(sz)]
        L.orth_orthogonalize_vjp_batched.argtypes = [P(orth_vjp_mat), i32, P(orth_bjorck_opts), vp, sz, vp, vp]
        L.orth_orthogonalize_save_workspace_size.argtypes = [P(orth_mat), i32, P(orth_bjorck_opts), P(sz)]
        L.orth_orthogonalize_save_batched.argtypes = [P(orth_mat), i32, P(orth_bjorck_opts), vp, sz, vp, vp]
        L.orth_aoc_param_shapes.argtypes = [P(orth_conv_geom)] + [P(i32)] * 5
        L.orth_build_conv_kernels_workspace_size.argtypes = [P(orth_conv_desc), i32, i32, P(sz)]
        L.orth_build_conv_kernels_batched.argtypes = [P(orth_conv_desc), i32, i32, vp, sz, vp]
        L.orth_build_conv_kernel.argtypes = [vp, vp, i32, i32, i32, i32, i32, i32, i32, vp, vp, sz, vp]
        L.orth_build_conv_kernels_vjp_workspace_size.argtypes = [P(orth_conv_vjp_desc), i32, i32, P(sz)]
        L.orth_build_conv_kernels_vjp_batched.argtypes = [P(orth_conv_vjp_desc), i32, i32, vp, sz, vp]
        L.orth_build_conv_kernels_save_workspace_size.argtypes = [P(orth_conv_desc), i32, i32, P(sz)]
        L.orth_build_conv_kernels_save_batched.argtypes = [P(orth_conv_desc), i32, i32, vp, sz, vp]
        L.orth_build_conv_kernels_vjp_saved_batched.argtypes = [P(orth_conv_vjp_desc), i32, i32, vp, sz, vp]
        L.orth_conv_apply.argtypes = [P(orth_conv_apply_args), vp]
        L.orth_exp_map_workspace_size.argtypes = [P(orth_mat), i32, P(orth_exp_opts), P(sz)]
        L.orth_exp_map_batched.argtypes = [P(orth_mat), i32, P(orth_exp_opts), vp, sz, vp, vp]
        L.orth_conv_exp_workspace_size.argtypes = [P(orth_conv_exp_desc), i32, i32, P(sz)]
        L.orth_conv_exp_batched.argtypes = [P(orth_conv_exp_desc), i32, i32, vp, sz, vp]
        L.orth_check_workspace_size.argtypes = [P(orth_check_args), P(sz)]
        L.orth_check_norm.argtypes = [P(orth_check_args), vp, vp, sz, vp]
        L.orth_status_string.argtypes = [ctypes.c_int]
        L.orth_status_string.restype = ctypes.c_char_p
        L.orth_last_error.restype = ctypes.c_char_p
        L.orth_timing_enable.argtypes = [i32]
        L.orth_timing_read.argtypes = [ctypes.c_char_p, P(ctypes.c_double), P(ctypes.c_int64)]
        L.orth_timing_filter.argtypes = [ctypes.c_char_p]
        L.orth_timing_span.argtypes = [ctypes.c_char_p, P(ctypes.c_double), P(ctypes.c_int64)]
        L.orth_timing_names.argtypes = [ctypes.c_char_p, sz]
        for name in EXPORTED:
            if name not in ("orth_status_string", "orth_last_error"):
                getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def _check(rc, where):
    if rc != ORTH_OK:
        raise OrthError(rc, where)


def _dtype_code(t):
    if t.dtype == torch.float32:
        return ORTH_F32
    if t.dtype == torch.bfloat16:
        return ORTH_BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _stream(stream):
    if stream is None:
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else stream)


def _ld(t):
    if t.dim() != 2 or t.stride(1) != 1:
        raise ValueError("matrices must be 2-D with unit column stride")
    return t.stride(0)


def _workspace(nbytes, device, workspace):
    if nbytes == 0:
        return None, 0
    if workspace is not None and workspace.numel() * workspace.element_size() >= nbytes:
        return workspace, workspace.numel() * workspace.element_size()
    ws = torch.empty(nbytes, dtype=torch.uint8, device=device)
    return ws, nbytes


def _mats(ins, outs):
    arr = (orth_mat * len(ins))()
    for i, (a, b) in enumerate(zip(ins, outs)):
        if a.shape != b.shape:
            raise ValueError("input and output shapes differ")
        arr[i] = orth_mat(a.data_ptr(), b.data_ptr(), a.shape[0], a.shape[1], _ld(a), _ld(b))
    return arr


def _opts(ins, outs, iters, beta, prescale, compute, power_iters=1, u=None, tile=0, saved=0, need_u=True):
    in_dt = _dtype_code(ins[0]) if ins else ORTH_F32
    out_dt = _dtype_code(outs[0]) if outs else ORTH_F32
    for a, b in zip(ins, outs):
        if _dtype_code(a) != in_dt or _dtype_code(b) != out_dt:
            raise TypeError("all inputs (and all outputs) must share one dtype")
    pres = {"frobenius": ORTH_PRESCALE_FROBENIUS, "none": ORTH_PRESCALE_NONE,
            "spectral": ORTH_PRESCALE_SPECTRAL}[prescale]
    comp = {"f32": ORTH_COMPUTE_F32, "bf16": ORTH_COMPUTE_BF16}[compute]
    uptr = None
    if pres == ORTH_PRESCALE_SPECTRAL and ins and (need_u or u is not None):
        need = sum(min(t.shape[0], t.shape[1]) for t in ins)
        if u is None or u.dtype != torch.float32 or not u.is_contiguous() or u.numel() < need:
            raise ValueError(f"spectral pre-scaling needs u: a contiguous float32 tensor of {need} values "
                             "(min(rows, cols) per matrix, packed in batch order)")
        uptr = u.data_ptr()
    return orth_bjorck_opts(iters, beta, pres, in_dt, out_dt, comp, power_iters, uptr, tile, saved)


def orth_orthogonalize_workspace_size(ins, iters, beta=0.5, prescale="frobenius", compute="f32", outs=None,
                                      power_iters=1, u=None, tile=0):
    outs = ins if outs is None else outs
    mats = _mats(ins, outs)
    opts = _opts(ins, outs, iters, beta, prescale, compute, power_iters, u, tile)
    n = ctypes.c_size_t()
    _check(lib().orth_orthogonalize_workspace_size(mats, len(ins), ctypes.byref(opts), ctypes.byref(n)),
           "orth_orthogonalize_workspace_size")
    return n.value


def orth_orthogonalize_batched(ins, outs, iters, beta=0.5, prescale="frobenius", compute="f32", status=None,
                               workspace=None, stream=None, power_iters=1, u=None, tile=0):
    """Björck-orthogonalize every ins[i] into outs[i] (see include/orth.h).
    prescale="spectral" takes power_iters and u, the packed float32 cached
    vectors (min(rows, cols) per matrix), updated in place.  tile (0, 128
    or 256) is the bf16 tile edge of matrices with min(rows, cols) >= 1024
    (0: chosen by occupancy).
    Returns the workspace tensor so that callers can reuse it."""
    mats = _mats(ins, outs)
    opts = _opts(ins, outs, iters, beta, prescale, compute, power_iters, u, tile)
    n = ctypes.c_size_t()
    _check(lib().orth_orthogonalize_workspace_size(mats, len(ins), ctypes.byref(opts), ctypes.byref(n)),
           "orth_orthogonalize_workspace_size")
    device = ins[0].device if ins else torch.device("cuda")
    ws, nbytes = _workspace(n.value, device, workspace)
    if status is not None and (status.dtype != torch.int32 or status.numel() < len(ins)):
        raise ValueError("status must be an int32 tensor with one slot per matrix")
    rc = lib().orth_orthogonalize_batched(mats, len(ins), ctypes.byref(opts),
                                          ws.data_ptr() if ws is not None else None, nbytes,
                                          status.data_ptr() if status is not None else None, _stream(stream))
    _check(rc, "orth_orthogonalize_batched")
    return ws


def orth_orthogonalize_batched_noalloc(ins, outs, iters, beta=0.5, prescale="frobenius", compute="f32",
                                       status=None, stream=None, power_iters=1, u=None, tile=0):
    """orth_orthogonalize_batched without a workspace: the library's own
    device scratch (ORTH_NOALLOC_SCRATCH_BYTES per GPU) holds the iterates,
    so neither the library nor this binding allocates anything.  Calls on
    one GPU share the scratch and must not overlap."""
    mats = _mats(ins, outs)
    opts = _opts(ins, outs, iters, beta, prescale, compute, power_iters, u, tile)
    if status is not None and (status.dtype != torch.int32 or status.numel() < len(ins)):
        raise ValueError("status must be an int32 tensor with one slot per matrix")
    rc = lib().orth_orthogonalize_batched_noalloc(mats, len(ins), ctypes.byref(opts),
                                                  status.data_ptr() if status is not None else None,
                                                  _stream(stream))
    _check(rc, "orth_orthogonalize_batched_noalloc")


def _vjp_mats(ws, gouts, gins):
    arr = (orth_vjp_mat * len(ws))()
    for i, (w, go, gi) in enumerate(zip(ws, gouts, gins)):
        if not (w.shape == go.shape == gi.shape):
            raise ValueError("w, grad_out and grad_in shapes differ")
        arr[i] = orth_vjp_mat(w.data_ptr(), go.data_ptr(), gi.data_ptr(), w.shape[0], w.shape[1], _ld(w), _ld(go),
                              _ld(gi))
    return arr


def orth_orthogonalize_vjp_batched(ws, grads_out, grads_in, iters, beta=0.5, prescale="frobenius", compute="f32",
                                   status=None, workspace=None, stream=None, tile=0, saved=False, power_iters=1,
                                   u=None):
    """dL/dW into grads_in[i] for L depending on ws[i] through
    orth_orthogonalize_batched with the same options, given grads_out[i] =
    dL/d(output) (see include/orth.h).  grads_in share the dtype of ws,
    grads_out that of the forward outputs.  saved=True takes the forward
    iterates from `workspace`, which orth_orthogonalize_save_batched filled
    for the same ws and options.  prescale="spectral": u holds the cached
    vectors as the differentiated forward found them (read only; not needed
    with saved=True).  Returns the workspace tensor."""
    if saved and workspace is None:
        raise ValueError("saved=True needs the workspace of orth_orthogonalize_save_batched")
    if len(ws) != len(grads_out) or len(ws) != len(grads_in):
        raise ValueError("ws, grads_out and grads_in must have the same length")
    for w, gi in zip(ws, grads_in):
        if w.dtype != gi.dtype:
            raise TypeError("grads_in must have the dtype of ws")
    mats = _vjp_mats(ws, grads_out, grads_in)
    opts = _opts(ws, grads_out, iters, beta, prescale, compute, power_iters, u, tile=tile, saved=1 if saved else 0,
                 need_u=not saved)
    n = ctypes.c_size_t()
    _check(lib().orth_orthogonalize_vjp_workspace_size(mats, len(ws), ctypes.byref(opts), ctypes.byref(n)),
           "orth_orthogonalize_vjp_workspace_size")
    device = ws[0].device if ws else torch.device("cuda")
    wsp, nbytes = _workspace(n.value, device, workspace)
    if status is not None and (status.dtype != torch.int32 or status.numel() < len(ws)):
        raise ValueError("status must be an int32 tensor with one slot per matrix")
    rc = lib().orth_orthogonalize_vjp_batched(mats, len(ws), ctypes.byref(opts),
                                              wsp.data_ptr() if wsp is not None else None, nbytes,
                                              status.data_ptr() if status is not None else None, _stream(stream))
    _check(rc, "orth_orthogonalize_vjp_batched")
    return wsp


def orth_orthogonalize_save_batched(ins, outs, iters, beta=0.5, prescale="frobenius", compute="f32", status=None,
                                    workspace=None, stream=None, tile=0, power_iters=1, u=None):
    """orth_orthogonalize_batched that also keeps, in the returned workspace,
    the forward iterates that orth_orthogonalize_vjp_batched(..., saved=True,
    workspace=<it>) reuses (see include/orth.h).  outs must not be ins."""
    mats = _mats(ins, outs)
    opts = _opts(ins, outs, iters, beta, prescale, compute, power_iters, u, tile=tile)
    n = ctypes.c_size_t()
    _check(lib().orth_orthogonalize_save_workspace_size(mats, len(ins), ctypes.byref(opts), ctypes.byref(n)),
           "orth_orthogonalize_save_workspace_size")
    device = ins[0].device if ins else torch.device("cuda")
    ws, nbytes = _workspace(n.value, device, workspace)
    if status is not None and (status.dtype != torch.int32 or status.numel() < len(ins)):
        raise ValueError("status must be an int32 tensor with one slot per matrix")
    rc = lib().orth_orthogonalize_save_batched(mats, len(ins), ctypes.byref(opts),
                                               ws.data_ptr() if ws is not None else None, nbytes,
                                               status.data_ptr() if status is not None else None, _stream(stream))
    _check(rc, "orth_orthogonalize_save_batched")
    return ws


def orth_orthogonalize_vjp_workspace_size(ws, iters, beta=0.5, prescale="frobenius", compute="f32",
                                          grads_out=None, tile=0, power_iters=1):
    grads_out = ws if grads_out is None else grads_out
    mats = _vjp_mats(ws, grads_out, ws)
    opts = _opts(ws, grads_out, iters, beta, prescale, compute, power_iters, tile=tile, need_u=False)
    n = ctypes.c_size_t()
    _check(lib().orth_orthogonalize_vjp_workspace_size(mats, len(ws), ctypes.byref(opts), ctypes.byref(n)),
           "orth_orthogonalize_vjp_workspace_size")
    return n.value


def orth_aoc_param_shapes(cin, cout, k, stride=1, dilation=1, groups=1):
    g = orth_conv_geom(cin, cout, k, stride, dilation, groups)
    out = [ctypes.c_int32() for _ in range(5)]
    _check(lib().orth_aoc_param_shapes(ctypes.byref(g), *[ctypes.byref(o) for o in out]), "orth_aoc_param_shapes")
    return tuple(o.value for o in out)


def _conv_descs(layers):
    arr = (orth_conv_desc * len(layers))()
    for i, L in enumerate(layers):
        geom = orth_conv_geom(*L["geom"])
        proj = L.get("proj")
        arr[i] = orth_conv_desc(geom, L["rko"].data_ptr(), proj.data_ptr() if proj is not None else None,
                                L["kernel"].data_ptr())
    return arr


def orth_build_conv_kernels_batched(layers, workspace=None, stream=None):
    """layers: list of dicts with geom=(cin, cout, k, stride, dilation, groups),
    rko, proj (or None) and kernel tensors (contiguous, one dtype)."""
    if not layers:
        return None
    dt = _dtype_code(layers[0]["kernel"])
    for L in layers:
        for key in ("rko", "proj", "kernel"):
            t = L.get(key)
            if t is not None and (not t.is_contiguous() or _dtype_code(t) != dt):
                raise ValueError(f"{key} must be contiguous and of the kernel's dtype")
    descs = _conv_descs(layers)
    n = ctypes.c_size_t()
    _check(lib().orth_build_conv_kernels_workspace_size(descs, len(layers), dt, ctypes.byref(n)),
           "orth_build_conv_kernels_workspace_size")
    ws, nbytes = _workspace(n.value, layers[0]["kernel"].device, workspace)
    rc = lib().orth_build_conv_kernels_batched(descs, len(layers), dt, ws.data_ptr() if ws is not None else None,
                                               nbytes, _stream(stream))
    _check(rc, "orth_build_conv_kernels_batched")
    return ws


def orth_build_conv_kernel(rko, proj, cin, cout, k, stride, dilation, groups, kernel_out, workspace=None,
                           stream=None):
    return orth_build_conv_kernels_batched(
        [dict(geom=(cin, cout, k, stride, dilation, groups), rko=rko, proj=proj, kernel=kernel_out)],
        workspace, stream)


def orth_build_conv_kernels_vjp_batched(layers, workspace=None, stream=None, saved=False):
    """layers: list of dicts with geom, rko, proj (or None), grad_kernel,
    grad_rko and grad_proj (or None) tensors (contiguous, one dtype).
    Writes dL/d rko and dL/d proj given dL/d kernel.  saved=True skips the
    forward recomputation: `workspace` holds what
    orth_build_conv_kernels_save_batched left for the same layers."""
    if not layers:
        return None
    if saved and workspace is None:
        raise ValueError("saved=True needs the workspace of orth_build_conv_kernels_save_batched")
    dt = _dtype_code(layers[0]["grad_kernel"])
    arr = (orth_conv_vjp_desc * len(layers))()
    for i, L in enumerate(layers):
        for key in ("rko", "proj", "grad_kernel", "grad_rko", "grad_proj"):
            t = L.get(key)
            if t is not None and (not t.is_contiguous() or _dtype_code(t) != dt):
                raise ValueError(f"{key} must be contiguous and of one dtype")
        ptr = lambda key: L[key].data_ptr() if L.get(key) is not None else None
        arr[i] = orth_conv_vjp_desc(orth_conv_geom(*L["geom"]), ptr("rko"), ptr("proj"), ptr("grad_kernel"),
                                    ptr("grad_rko"), ptr("grad_proj"))
    n = ctypes.c_size_t()
    _check(lib().orth_build_conv_kernels_vjp_workspace_size(arr, len(layers), dt, ctypes.byref(n)),
           "orth_build_conv_kernels_vjp_workspace_size")
    ws, nbytes = _workspace(n.value, layers[0]["grad_kernel"].device, workspace)
    fn = lib().orth_build_conv_kernels_vjp_saved_batched if saved else lib().orth_build_conv_kernels_vjp_batched
    rc = fn(arr, len(layers), dt, ws.data_ptr() if ws is not None else None, nbytes, _stream(stream))
    _check(rc, "orth_build_conv_kernels_vjp_batched")
    return ws


def orth_build_conv_kernels_save_batched(layers, workspace=None, stream=None):
    """orth_build_conv_kernels_batched that also keeps, in the returned
    (composition-VJP) workspace, what orth_build_conv_kernels_vjp_batched(...,
    saved=True, workspace=<it>) reuses.  layers as for
    orth_build_conv_kernels_batched."""
    if not layers:
        return None
    dt = _dtype_code(layers[0]["kernel"])
    for L in layers:
        for key in ("rko", "proj", "kernel"):
            t = L.get(key)
            if t is not None and (not t.is_contiguous() or _dtype_code(t) != dt):
                raise ValueError(f"{key} must be contiguous and of the kernel's dtype")
    descs = _conv_descs(layers)
    n = ctypes.c_size_t()
    _check(lib().orth_build_conv_kernels_save_workspace_size(descs, len(layers), dt, ctypes.byref(n)),
           "orth_build_conv_kernels_save_workspace_size")
    ws, nbytes = _workspace(n.value, layers[0]["kernel"].device, workspace)
    rc = lib().orth_build_conv_kernels_save_batched(descs, len(layers), dt, ws.data_ptr() if ws is not None else None,
                                                    nbytes, _stream(stream))
    _check(rc, "orth_build_conv_kernels_save_batched")
    return ws


def orth_conv_apply(kernel, geom, x, transposed=False, stream=None):
    """Circular conv (or its transpose) of the float32 NCHW batch x with the
    explicit kernel; returns the new output tensor."""
    if x.dtype != torch.float32 or not x.is_contiguous() or not kernel.is_contiguous():
        raise ValueError("x must be contiguous float32 and the kernel contiguous")
    cin, cout, k, s, d, g = geom
    b = x.shape[0]
    if transposed:
        h, w = x.shape[2] * s, x.shape[3] * s
        y = torch.empty(b, cin, h, w, dtype=torch.float32, device=x.device)
    else:
        h, w = x.shape[2], x.shape[3]
        y = torch.empty(b, cout, h // s, w // s, dtype=torch.float32, device=x.device)
    args = orth_conv_apply_args(orth_conv_geom(*geom), kernel.data_ptr(), _dtype_code(kernel), int(transposed),
                                x.data_ptr(), y.data_ptr(), b, h, w)
    _check(lib().orth_conv_apply(ctypes.byref(args), _stream(stream)), "orth_conv_apply")
    return y


def orth_exp_map_batched(ins, outs, terms, u, power_iters=1, status=None, workspace=None, stream=None):
    """What = exp(A / sigma), A = W - W^T, for every square ins[i] into
    outs[i] (see include/orth.h); u: packed float32 cached vectors (C per
    matrix), updated in place.  Returns the workspace tensor."""
    if not ins:
        return None
    mats = _mats(ins, outs)
    in_dt, out_dt = _dtype_code(ins[0]), _dtype_code(outs[0])
    for a, b in zip(ins, outs):
        if _dtype_code(a) != in_dt or _dtype_code(b) != out_dt:
            raise TypeError("all inputs (and all outputs) must share one dtype")
    need = sum(t.shape[0] for t in ins)
    if u.dtype != torch.float32 or not u.is_contiguous() or u.numel() < need:
        raise ValueError(f"u must be a contiguous float32 tensor of {need} values")
    opts = orth_exp_opts(terms, power_iters, u.data_ptr(), in_dt, out_dt)
    n = ctypes.c_size_t()
    _check(lib().orth_exp_map_workspace_size(mats, len(ins), ctypes.byref(opts), ctypes.byref(n)),
           "orth_exp_map_workspace_size")
    ws, nbytes = _workspace(n.value, ins[0].device, workspace)
    if status is not None and (status.dtype != torch.int32 or status.numel() < len(ins)):
        raise ValueError("status must be an int32 tensor with one slot per matrix")
    rc = lib().orth_exp_map_batched(mats, len(ins), ctypes.byref(opts), ws.data_ptr() if ws is not None else None,
                                    nbytes, status.data_ptr() if status is not None else None, _stream(stream))
    _check(rc, "orth_exp_map_batched")
    return ws


def orth_conv_exp_batched(layers, workspace=None, stream=None):
    """layers: dicts with kernel (c x c x k x k), out (c x c x S x S,
    S = terms (k - 1) + 1), terms and scale; contiguous, one dtype."""
    if not layers:
        return None
    dt = _dtype_code(layers[0]["kernel"])
    arr = (orth_conv_exp_desc * len(layers))()
    for i, L in enumerate(layers):
        kern, out = L["kernel"], L["out"]
        if not kern.is_contiguous() or not out.is_contiguous() or _dtype_code(kern) != dt or _dtype_code(out) != dt:
            raise ValueError("kernel and out must be contiguous and of one dtype")
        c, k = kern.shape[0], kern.shape[2]
        arr[i] = orth_conv_exp_desc(c, k, L["terms"], float(L.get("scale", 1.0)), kern.data_ptr(), out.data_ptr())
    n = ctypes.c_size_t()
    _check(lib().orth_conv_exp_workspace_size(arr, len(layers), dt, ctypes.byref(n)), "orth_conv_exp_workspace_size")
    ws, nbytes = _workspace(n.value, layers[0]["kernel"].device, workspace)
    rc = lib().orth_conv_exp_batched(arr, len(layers), dt, ws.data_ptr() if ws is not None else None, nbytes,
                                     _stream(stream))
    _check(rc, "orth_conv_exp_batched")
    return ws


def _check_call(args, out, workspace, stream):
    n = ctypes.c_size_t()
    _check(lib().orth_check_workspace_size(ctypes.byref(args), ctypes.byref(n)), "orth_check_workspace_size")
    ws, nbytes = _workspace(n.value, out.device, workspace)
    rc = lib().orth_check_norm(ctypes.byref(args), out.data_ptr(), ws.data_ptr() if ws is not None else None,
                               nbytes, _stream(stream))
    _check(rc, "orth_check_norm")


def orth_check_norm_gram(mats, workspace=None, stream=None):
    """max |G - I| per matrix (G the smaller Gram matrix), as a float32 tensor."""
    arr = _mats(mats, mats)
    out = torch.empty(len(mats), dtype=torch.float32, device=mats[0].device)
    args = orth_check_args()
    args.mode = ORTH_CHECK_GRAM
    args.mats = ctypes.cast(arr, ctypes.POINTER(orth_mat))
    args.n_mats = len(mats)
    args.mat_dtype = _dtype_code(mats[0])
    _check_call(args, out, workspace, stream)
    return out


def orth_check_norm_conv(kernel, geom, x, adjoint=False, workspace=None, stream=None):
    """||conv_circ(K, x_b)|| / ||x_b|| per sample (or the adjoint's ratio)."""
    if x.dtype != torch.float32 or not x.is_contiguous() or not kernel.is_contiguous():
        raise ValueError("x must be contiguous float32 and the kernel contiguous")
    out = torch.empty(x.shape[0], dtype=torch.float32, device=x.device)
    args = orth_check_args()
    args.mode = ORTH_CHECK_CONV_ADJOINT if adjoint else ORTH_CHECK_CONV
    args.kernel = kernel.data_ptr()
    args.kernel_dtype = _dtype_code(kernel)
    args.geom = orth_conv_geom(*geom)
    args.x = x.data_ptr()
    args.batch, args.height, args.width = x.shape[0], x.shape[2], x.shape[3]
    _check_call(args, out, workspace, stream)
    return out


def orth_timing_enable(on=True):
    _check(lib().orth_timing_enable(1 if on else 0), "orth_timing_enable")


def orth_timing_filter(*prefixes):
    """Time only launches whose kernel names start with one of the prefixes
    (none: every launch)."""
    _check(lib().orth_timing_filter(";".join(prefixes).encode()), "orth_timing_filter")


def orth_timing_reset():
    _check(lib().orth_timing_reset(), "orth_timing_reset")


def orth_timing_read(name):
    ms, n = ctypes.c_double(), ctypes.c_int64()
    _check(lib().orth_timing_read(name.encode(), ctypes.byref(ms), ctypes.byref(n)), "orth_timing_read")
    return ms.value, n.value


def orth_timing_span(*prefixes):
    """Wall-clock ms covered by the launches whose names start with any of
    the prefixes (overlapping launches count once), and their number."""
    ms, n = ctypes.c_double(), ctypes.c_int64()
    _check(lib().orth_timing_span(";".join(prefixes).encode(), ctypes.byref(ms), ctypes.byref(n)),
           "orth_timing_span")
    return ms.value, n.value


def orth_timing_names():
    buf = ctypes.create_string_buffer(4096)
    _check(lib().orth_timing_names(buf, 4096), "orth_timing_names")
    return [s for s in buf.value.decode().split(";") if s]
