"""Thin Python binding of the WBMM C ABI (include/wbmm.h).

Argument marshalling only: tensors are handed to libwbmm.so as raw device
pointers together with torch's current HIP stream; every step of the operator
runs in the library's HIP kernels.  There is no fallback: if libwbmm.so is not
built, or a call fails, an exception is raised.

Names follow the C entry points: ``wbmm_forward``, ``wbmm_backward_input``,
``wbmm_backward_table``, ``wbmm_backward_table_workspace_bytes``,
``wbmm_backward``, ``wbmm_backward_workspace_bytes``, the hierarchical form
``wbmm_hier_forward``, ``wbmm_hier_backward_input``, ``wbmm_hier_backward``,
``wbmm_hier_backward_workspace_bytes``, the cached-matrix form
``wbmm_build_matrix``, ``wbmm_dense_forward``, ``wbmm_dense_backward_input``,
``wbmm_dense_backward_matrix``, ``wbmm_bin_matrix``, and
``wbmm_relative_index``, ``wbmm_status_string``.  ``wbmm_rect_*`` compose the
cached-matrix calls into WBMM for rectangular windows.
"""
from __future__ import annotations

import ctypes
import os

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libwbmm.so")

WBMM_OK = 0
WBMM_ERR_INVALID_ARG = 1
WBMM_ERR_UNSUPPORTED = 2
WBMM_ERR_HIP = 3
WBMM_ERR_SCRATCH = 4
NOALLOC_SCRATCH_BYTES = 4 << 20  # WBMM_NOALLOC_SCRATCH_BYTES of include/wbmm.h

DTYPE_CODES = {torch.float32: 0, torch.bfloat16: 1, torch.float16: 2}

EXPORTED = ("wbmm_forward", "wbmm_backward_input", "wbmm_backward_table",
            "wbmm_backward_table_workspace_bytes", "wbmm_backward",
            "wbmm_backward_workspace_bytes", "wbmm_backward_noalloc", "wbmm_hier_forward",
            "wbmm_hier_backward_input", "wbmm_hier_backward",
            "wbmm_hier_backward_workspace_bytes", "wbmm_build_matrix",
            "wbmm_dense_forward", "wbmm_dense_backward_input",
            "wbmm_dense_backward_matrix", "wbmm_bin_matrix", "wbmm_status_string",
            "wbmm_relative_index", "wbmm_version")

_lib = None


class WbmmError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__("%s: %s" % (what, wbmm_status_string(status)))


def load_library(path: str = LIB_PATH):
    """Load libwbmm.so and declare its signatures.  Raises if it is missing."""
    global _lib
    if _lib is not None and path == LIB_PATH:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError("libwbmm.so is not built (%s); run `python -m "
                           "paper_2607_02097_amd.build` first" % path)
    lib = ctypes.CDLL(path)
    vp, i64, ci, st = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_int
    shape = [i64, i64, i64, i64, ci, ci, vp]
    lib.wbmm_forward.argtypes = [vp, vp, vp] + shape
    lib.wbmm_forward.restype = st
    lib.wbmm_backward_input.argtypes = [vp, vp, vp] + shape
    lib.wbmm_backward_input.restype = st
    lib.wbmm_backward_table_workspace_bytes.argtypes = [i64, i64, i64, i64, ci, ci]
    lib.wbmm_backward_table_workspace_bytes.restype = ctypes.c_size_t
    lib.wbmm_backward_table.argtypes = [vp, vp, vp, vp, ctypes.c_size_t] + shape
    lib.wbmm_backward_table.restype = st
    lib.wbmm_backward_workspace_bytes.argtypes = [i64, i64, i64, i64, ci, ci]
    lib.wbmm_backward_workspace_bytes.restype = ctypes.c_size_t
    lib.wbmm_backward.argtypes = [vp, vp, vp, vp, vp, vp, ctypes.c_size_t] + shape
    lib.wbmm_backward.restype = st
    lib.wbmm_backward_noalloc.argtypes = [vp, vp, vp, vp, vp] + shape
    lib.wbmm_backward_noalloc.restype = st
    lib.wbmm_hier_forward.argtypes = [vp, vp, vp, vp] + shape
    lib.wbmm_hier_forward.restype = st
    lib.wbmm_hier_backward_input.argtypes = [vp, vp, vp, vp] + shape
    lib.wbmm_hier_backward_input.restype = st
    lib.wbmm_hier_backward_workspace_bytes.argtypes = [i64, i64, i64, i64, ci, ci]
    lib.wbmm_hier_backward_workspace_bytes.restype = ctypes.c_size_t
    lib.wbmm_hier_backward.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, ctypes.c_size_t] + shape
    lib.wbmm_hier_backward.restype = st
    dshape = [i64, i64, i64, i64, ci, ci, ci, vp]
    lib.wbmm_build_matrix.argtypes = [vp, vp, i64, ci, ci, ci, vp]
    lib.wbmm_build_matrix.restype = st
    lib.wbmm_dense_forward.argtypes = [vp, vp, vp] + dshape
    lib.wbmm_dense_forward.restype = st
    lib.wbmm_dense_backward_input.argtypes = [vp, vp, vp] + dshape
    lib.wbmm_dense_backward_input.restype = st
    lib.wbmm_dense_backward_matrix.argtypes = [vp, vp, vp] + dshape
    lib.wbmm_dense_backward_matrix.restype = st
    lib.wbmm_bin_matrix.argtypes = [vp, vp, i64, ci, ci, vp]
    lib.wbmm_bin_matrix.restype = st
    lib.wbmm_status_string.argtypes = [st]
    lib.wbmm_status_string.restype = ctypes.c_char_p
    lib.wbmm_relative_index.argtypes = [ci, ctypes.POINTER(ctypes.c_int32)]
    lib.wbmm_relative_index.restype = st
    lib.wbmm_version.argtypes = []
    lib.wbmm_version.restype = ctypes.c_char_p
    if path == LIB_PATH:
        _lib = lib
    return lib


def wbmm_status_string(status: int) -> str:
    return load_library().wbmm_status_string(int(status)).decode()


def _stream(t: torch.Tensor, stream):
    if stream is None:
        return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)
    if isinstance(stream, torch.cuda.Stream):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def _check_tensor(t: torch.Tensor, name: str):
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if t.device.type != "cuda":
        raise ValueError("%s must be a GPU tensor (got %s)" % (name, t.device))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)


def _code(dtype) -> int:
    if dtype not in DTYPE_CODES:
        raise TypeError("unsupported dtype %s (float32, bfloat16, float16)" % dtype)
    return DTYPE_CODES[dtype]


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr())


def _forward_like(fn_name, src, table, w, out, stream):
    _check_tensor(src, "input")
    _check_tensor(table, "table")
    if src.dim() != 4:
        raise ValueError("input must be [B, C, H, W]")
    B, C, H, W = src.shape
    if table.dtype != src.dtype or table.device != src.device:
        raise ValueError("table must match the input's dtype and device")
    if out is None:
        out = torch.empty_like(src)
    else:
        _check_tensor(out, "out")
        if out.shape != src.shape or out.dtype != src.dtype or out.device != src.device:
            raise ValueError("out must match the input's shape, dtype and device")
    with torch.cuda.device(src.device):
        st = getattr(load_library(), fn_name)(_ptr(src), _ptr(table), _ptr(out), B, C, H, W,
                                              int(w), _code(src.dtype), _stream(src, stream))
    if st != WBMM_OK:
        raise WbmmError(st, fn_name)
    return out


def wbmm_forward(x: torch.Tensor, table: torch.Tensor, w: int, out=None, stream=None):
    """y = WBMM(x; table, w).  x [B,C,H,W], table [C,(2w-1)^2], same dtype."""
    return _forward_like("wbmm_forward", x, table, w, out, stream)


def wbmm_backward_input(dy: torch.Tensor, table: torch.Tensor, w: int, out=None, stream=None):
    """dx for upstream gradient dy (per window dx = dy M^T)."""
    return _forward_like("wbmm_backward_input", dy, table, w, out, stream)


def wbmm_backward_table_workspace_bytes(shape, w: int, dtype) -> int:
    B, C, H, W = shape
    return int(load_library().wbmm_backward_table_workspace_bytes(B, C, H, W, int(w), _code(dtype)))


_WS_CACHE = {}


def _torch_stream(device, stream):
    """The torch stream object of the stream a call is enqueued on."""
    if stream is None:
        return torch.cuda.current_stream(device)
    if isinstance(stream, torch.cuda.Stream):
        return stream
    return torch.cuda.ExternalStream(int(stream), device=device)


def _cached_workspace(device, nbytes, stream, shape_key):
    """A workspace kept per (device, stream, call shape).  The library writes
    the partial sums it holds before reading them, so its contents on entry
    do not matter; it is allocated on the stream the call is enqueued on."""
    ts = _torch_stream(device, stream)
    key = (str(device), ts.cuda_stream, shape_key)
    ws = _WS_CACHE.get(key)
    if ws is None:
        with torch.cuda.stream(ts):
            ws = torch.empty(nbytes, dtype=torch.uint8, device=device)
        _WS_CACHE[key] = ws
    return ws


def new_workspace(nbytes: int, device="cuda") -> torch.Tensor:
    """A workspace for wbmm_backward_table / wbmm_backward (see
    include/wbmm.h); any contents."""
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


def wbmm_backward_table(x: torch.Tensor, dy: torch.Tensor, w: int, out=None, workspace=None,
                        stream=None):
    """dtable (float32 [C,(2w-1)^2], overwritten) for input x and gradient dy.

    ``workspace``: a uint8 device tensor of at least
    wbmm_backward_table_workspace_bytes() bytes, any contents (see
    include/wbmm.h; ``new_workspace`` makes one).  When omitted, a workspace
    cached per (device, stream, shape) is used."""
    _check_tensor(x, "x")
    _check_tensor(dy, "dy")
    if dy.shape != x.shape or dy.dtype != x.dtype or dy.device != x.device:
        raise ValueError("dy must match x's shape, dtype and device")
    B, C, H, W = x.shape
    k = (2 * int(w) - 1) ** 2
    if out is None:
        out = torch.empty((C, k), dtype=torch.float32, device=x.device)
    else:
        _check_tensor(out, "out")
        if out.dtype != torch.float32 or out.numel() != C * k or out.device != x.device:
            raise ValueError("out must be float32 [C, (2w-1)^2] on x's device")
    need = wbmm_backward_table_workspace_bytes(x.shape, w, x.dtype)
    if workspace is None and need > 0:
        workspace = _cached_workspace(x.device, need, stream, (tuple(x.shape), int(w), x.dtype))
    ws_ptr = ctypes.c_void_p(workspace.data_ptr() if workspace is not None else 0)
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    with torch.cuda.device(x.device):
        st = load_library().wbmm_backward_table(_ptr(x), _ptr(dy), _ptr(out), ws_ptr, ws_bytes,
                                                B, C, H, W, int(w), _code(x.dtype),
                                                _stream(x, stream))
    if st != WBMM_OK:
        raise WbmmError(st, "wbmm_backward_table")
    return out


def wbmm_backward_workspace_bytes(shape, w: int, dtype) -> int:
    B, C, H, W = shape
    return int(load_library().wbmm_backward_workspace_bytes(B, C, H, W, int(w), _code(dtype)))


def wbmm_backward(x: torch.Tensor, dy: torch.Tensor, table: torch.Tensor, w: int, dx=None,
                  dtable=None, workspace=None, stream=None):
    """Both gradients in one pass: returns (dx, dtable), dx like x, dtable
    float32 [C,(2w-1)^2] (overwritten).  ``workspace`` as for
    ``wbmm_backward_table``."""
    _check_tensor(x, "x")
    _check_tensor(dy, "dy")
    _check_tensor(table, "table")
    if dy.shape != x.shape or dy.dtype != x.dtype or dy.device != x.device:
        raise ValueError("dy must match x's shape, dtype and device")
    if table.dtype != x.dtype or table.device != x.device:
        raise ValueError("table must match x's dtype and device")
    B, C, H, W = x.shape
    k = (2 * int(w) - 1) ** 2
    if dx is None:
        dx = torch.empty_like(x)
    else:
        _check_tensor(dx, "dx")
        if dx.shape != x.shape or dx.dtype != x.dtype or dx.device != x.device:
            raise ValueError("dx must match x's shape, dtype and device")
    if dtable is None:
        dtable = torch.empty((C, k), dtype=torch.float32, device=x.device)
    else:
        _check_tensor(dtable, "dtable")
        if dtable.dtype != torch.float32 or dtable.numel() != C * k or dtable.device != x.device:
            raise ValueError("dtable must be float32 [C, (2w-1)^2] on x's device")
    need = wbmm_backward_workspace_bytes(x.shape, w, x.dtype)
    if workspace is None and need > 0:
        workspace = _cached_workspace(x.device, need, stream, (tuple(x.shape), int(w), x.dtype))
    ws_ptr = ctypes.c_void_p(workspace.data_ptr() if workspace is not None else 0)
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    with torch.cuda.device(x.device):
        st = load_library().wbmm_backward(_ptr(x), _ptr(dy), _ptr(table), _ptr(dx), _ptr(dtable),
                                          ws_ptr, ws_bytes, B, C, H, W, int(w), _code(x.dtype),
                                          _stream(x, stream))
    if st != WBMM_OK:
        raise WbmmError(st, "wbmm_backward")
    return dx, dtable


def wbmm_backward_noalloc(x: torch.Tensor, dy: torch.Tensor, table: torch.Tensor, w: int, dx: torch.Tensor,
                          dtable: torch.Tensor, stream=None):
    """wbmm_backward without a workspace: the library's static scratch holds
    the table gradient's partial sums (see include/wbmm.h).  The
    caller passes the outputs; nothing is allocated."""
    for t, n in ((x, "x"), (dy, "dy"), (table, "table"), (dx, "dx"), (dtable, "dtable")):
        _check_tensor(t, n)
    if dy.shape != x.shape or dy.dtype != x.dtype or dx.shape != x.shape or dx.dtype != x.dtype:
        raise ValueError("dy and dx must match x's shape and dtype")
    if table.dtype != x.dtype or dtable.dtype != torch.float32:
        raise ValueError("table in x's dtype, dtable float32")
    B, C, H, W = x.shape
    with torch.cuda.device(x.device):
        st = load_library().wbmm_backward_noalloc(_ptr(x), _ptr(dy), _ptr(table), _ptr(dx), _ptr(dtable),
                                                  B, C, H, W, int(w), _code(x.dtype), _stream(x, stream))
    if st != WBMM_OK:
        raise WbmmError(st, "wbmm_backward_noalloc")
    return dx, dtable


def _hier_like(fn_name, src, tg, tl, wl, out, stream):
    _check_tensor(src, "input")
    _check_tensor(tg, "table_g")
    _check_tensor(tl, "table_l")
    if src.dim() != 4:
        raise ValueError("input must be [B, C, H, W]")
    B, C, H, W = src.shape
    for t in (tg, tl):
        if t.dtype != src.dtype or t.device != src.device:
            raise ValueError("tables must match the input's dtype and device")
    if out is None:
        out = torch.empty_like(src)
    else:
        _check_tensor(out, "out")
        if out.shape != src.shape or out.dtype != src.dtype or out.device != src.device:
            raise ValueError("out must match the input's shape, dtype and device")
    with torch.cuda.device(src.device):
        st = getattr(load_library(), fn_name)(_ptr(src), _ptr(tg), _ptr(tl), _ptr(out), B, C, H, W,
                                              int(wl), _code(src.dtype), _stream(src, stream))
    if st != WBMM_OK:
        raise WbmmError(st, fn_name)
    return out


def wbmm_hier_forward(x, table_g, table_l, wl: int, out=None, stream=None):
    """Hierarchical form: y = x M_fused per 2wl x 2wl window, table_g
    [C,(4wl-1)^2], table_l [C,(2wl-1)^2]."""
    return _hier_like("wbmm_hier_forward", x, table_g, table_l, wl, out, stream)


def wbmm_hier_backward_input(dy, table_g, table_l, wl: int, out=None, stream=None):
    """dx = dy M_fused^T of the hierarchical form."""
    return _hier_like("wbmm_hier_backward_input", dy, table_g, table_l, wl, out, stream)


def wbmm_hier_backward_workspace_bytes(shape, wl: int, dtype) -> int:
    B, C, H, W = shape
    return int(load_library().wbmm_hier_backward_workspace_bytes(B, C, H, W, int(wl), _code(dtype)))


def wbmm_hier_backward(x, dy, table_g, table_l, wl: int, workspace=None, stream=None):
    """All gradients of the hierarchical form: (dx, dtable_g, dtable_l), the
    table gradients float32."""
    _check_tensor(x, "x")
    _check_tensor(dy, "dy")
    if dy.shape != x.shape or dy.dtype != x.dtype or dy.device != x.device:
        raise ValueError("dy must match x's shape, dtype and device")
    B, C, H, W = x.shape
    dx = torch.empty_like(x)
    dtg = torch.empty((C, (4 * int(wl) - 1) ** 2), dtype=torch.float32, device=x.device)
    dtl = torch.empty((C, (2 * int(wl) - 1) ** 2), dtype=torch.float32, device=x.device)
    need = wbmm_hier_backward_workspace_bytes(x.shape, wl, x.dtype)
    if workspace is None and need > 0:
        workspace = _cached_workspace(x.device, need, stream, ("hier", tuple(x.shape), int(wl), x.dtype))
    ws_ptr = ctypes.c_void_p(workspace.data_ptr() if workspace is not None else 0)
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    with torch.cuda.device(x.device):
        st = load_library().wbmm_hier_backward(_ptr(x), _ptr(dy), _ptr(table_g), _ptr(table_l), _ptr(dx),
                                               _ptr(dtg), _ptr(dtl), ws_ptr, ws_bytes, B, C, H, W, int(wl),
                                               _code(x.dtype), _stream(x, stream))
    if st != WBMM_OK:
        raise WbmmError(st, "wbmm_hier_backward")
    return dx, dtg, dtl


# ------------------------------------------------ cached-matrix (dense) form

def _call(fn_name, dev, *args):
    with torch.cuda.device(dev):
        st = getattr(load_library(), fn_name)(*args)
    if st != WBMM_OK:
        raise WbmmError(st, fn_name)


def wbmm_build_matrix(table, wh: int, ww: int, out=None, stream=None):
    """M [C, d, d] (d = wh ww), M[c][i][j] = table[c][I(i, j)], in the
    table's dtype."""
    _check_tensor(table, "table")
    C = table.shape[0]
    d = int(wh) * int(ww)
    if out is None:
        out = torch.empty((C, d, d), dtype=table.dtype, device=table.device)
    else:
        _check_tensor(out, "out")
        if out.numel() != C * d * d or out.dtype != table.dtype or out.device != table.device:
            raise ValueError("out must be [C, d, d] in the table's dtype and device")
    _call("wbmm_build_matrix", table.device, _ptr(table), _ptr(out), C, int(wh), int(ww), _code(table.dtype),
          _stream(table, stream))
    return out


def _dense_like(fn_name, src, m, wh, ww, out, stream):
    _check_tensor(src, "input")
    _check_tensor(m, "m")
    B, C, H, W = src.shape
    d = int(wh) * int(ww)
    if m.dtype != src.dtype or m.device != src.device or m.numel() != C * d * d:
        raise ValueError("m must be [C, d, d] in the input's dtype and device")
    if out is None:
        out = torch.empty_like(src)
    else:
        _check_tensor(out, "out")
        if out.shape != src.shape or out.dtype != src.dtype or out.device != src.device:
            raise ValueError("out must match the input's shape, dtype and device")
    _call(fn_name, src.device, _ptr(src), _ptr(m), _ptr(out), B, C, H, W, int(wh), int(ww), _code(src.dtype),
          _stream(src, stream))
    return out


def wbmm_dense_forward(x, m, wh: int, ww: int, out=None, stream=None):
    """y_window = x_window m[c] per wh x ww window."""
    return _dense_like("wbmm_dense_forward", x, m, wh, ww, out, stream)


def wbmm_dense_backward_input(dy, m, wh: int, ww: int, out=None, stream=None):
    """dx_window = dy_window m[c]^T."""
    return _dense_like("wbmm_dense_backward_input", dy, m, wh, ww, out, stream)


def wbmm_dense_backward_matrix(x, dy, wh: int, ww: int, out=None, stream=None):
    """dm [C, d, d] float32: sum over windows of x_window^T dy_window."""
    _check_tensor(x, "x")
    _check_tensor(dy, "dy")
    if dy.shape != x.shape or dy.dtype != x.dtype or dy.device != x.device:
        raise ValueError("dy must match x's shape, dtype and device")
    B, C, H, W = x.shape
    d = int(wh) * int(ww)
    if out is None:
        out = torch.empty((C, d, d), dtype=torch.float32, device=x.device)
    _call("wbmm_dense_backward_matrix", x.device, _ptr(x), _ptr(dy), _ptr(out), B, C, H, W, int(wh), int(ww),
          _code(x.dtype), _stream(x, stream))
    return out


def wbmm_bin_matrix(dm, wh: int, ww: int, out=None, stream=None):
    """dtable [C, (2wh-1)(2ww-1)] float32 from a float32 matrix gradient."""
    _check_tensor(dm, "dm")
    if dm.dtype != torch.float32:
        raise TypeError("dm must be float32")
    C = dm.shape[0]
    k = (2 * int(wh) - 1) * (2 * int(ww) - 1)
    if out is None:
        out = torch.empty((C, k), dtype=torch.float32, device=dm.device)
    _call("wbmm_bin_matrix", dm.device, _ptr(dm), _ptr(out), C, int(wh), int(ww), _stream(dm, stream))
    return out


def wbmm_rect_forward(x, table, wh: int, ww: int, m=None, stream=None):
    """WBMM with wh x ww windows (table [C,(2wh-1)(2ww-1)]): the matrix is
    built (or ``m`` reused) and applied per window."""
    if m is None:
        m = wbmm_build_matrix(table, wh, ww, stream=stream)
    return wbmm_dense_forward(x, m, wh, ww, stream=stream)


def wbmm_rect_backward_input(dy, table, wh: int, ww: int, m=None, stream=None):
    if m is None:
        m = wbmm_build_matrix(table, wh, ww, stream=stream)
    return wbmm_dense_backward_input(dy, m, wh, ww, stream=stream)


def wbmm_rect_backward_table(x, dy, wh: int, ww: int, stream=None):
    """Table gradient with wh x ww windows (float32): the matrix gradient
    folded onto the table."""
    return wbmm_bin_matrix(wbmm_dense_backward_matrix(x, dy, wh, ww, stream=stream), wh, ww, stream=stream)


def wbmm_relative_index(w: int) -> torch.Tensor:
    """The int32 [d, d] index I of eq. index_computation (host tensor)."""
    d = int(w) * int(w)
    out = torch.empty((d, d), dtype=torch.int32)
    st = load_library().wbmm_relative_index(
        int(w), ctypes.cast(out.data_ptr(), ctypes.POINTER(ctypes.c_int32)))
    if st != WBMM_OK:
        raise WbmmError(st, "wbmm_relative_index")
    return out


def wbmm_version() -> str:
    return load_library().wbmm_version().decode()


class WBMMFunction(torch.autograd.Function):
    """Autograd composition of the entry points: the forward, then both
    gradients in one fused pass (or the one that is needed).  The table
    gradient is computed in float32 and cast to the table's dtype."""

    @staticmethod
    def forward(ctx, x, table, w):
        ctx.w = int(w)
        ctx.save_for_backward(x, table)
        return wbmm_forward(x.contiguous(), table.contiguous(), ctx.w)

    @staticmethod
    def backward(ctx, dy):
        x, table = ctx.saved_tensors
        dy = dy.contiguous()
        need_x, need_t = ctx.needs_input_grad[0], ctx.needs_input_grad[1]
        dx = dt = None
        if need_x and need_t:
            dx, dt = wbmm_backward(x, dy, table, ctx.w)
            dt = dt.to(table.dtype)
        elif need_x:
            dx = wbmm_backward_input(dy, table, ctx.w)
        elif need_t:
            dt = wbmm_backward_table(x, dy, ctx.w).to(table.dtype)
        return dx, dt, None


def wbmm(x, table, w):
    """Differentiable WBMM: y = WBMM(x; table, w)."""
    return WBMMFunction.apply(x, table, w)


class WBMMHierFunction(torch.autograd.Function):
    """Autograd of the hierarchical form (table gradients cast to the tables'
    dtype)."""

    @staticmethod
    def forward(ctx, x, table_g, table_l, wl):
        ctx.wl = int(wl)
        ctx.save_for_backward(x, table_g, table_l)
        return wbmm_hier_forward(x.contiguous(), table_g.contiguous(), table_l.contiguous(), ctx.wl)

    @staticmethod
    def backward(ctx, dy):
        x, tg, tl = ctx.saved_tensors
        dx, dtg, dtl = wbmm_hier_backward(x, dy.contiguous(), tg, tl, ctx.wl)
        return dx, dtg.to(tg.dtype), dtl.to(tl.dtype), None


def wbmm_hier(x, table_g, table_l, wl):
    """Differentiable hierarchical WBMM (global windows 2 wl, local wl)."""
    return WBMMHierFunction.apply(x, table_g, table_l, wl)
