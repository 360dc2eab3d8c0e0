"""WBMM oracle — TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.

Plain fp64 CPU reference of the Windowed Batch Matrix Multiplication operator
(Alg. 1, eq. index_computation / index_select, Theorem 3.2's row-vector
convention) and of its two backward passes (chain rule on the forward; the
paper only states that gradients flow through the table, Sec. 3.4.5).

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the HIP library
and never imports it; the product path never imports this package.

The arithmetic lives in ``wbmm_oracle.c`` (plain loops, one sequential fp64 sum
per output element, OpenMP across planes/channels only).  This module builds it
with gcc and marshals numpy float64 arrays through ctypes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import sys

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "wbmm_oracle.c")
LIB_PATH = os.path.join(_HERE, "libwbmm_oracle.so")

_lib = None


def build(mutant: int = 0, out_path: str | None = None, openmp: bool = True) -> str:
    """Compile the oracle with gcc (-O2 -fopenmp, strict IEEE: no fast-math,
    no FMA contraction so every product is rounded before it is summed).

    ``mutant`` selects one of the planted mistakes used by the test that shows
    the pins reject them (0 = the real oracle).  Planted-mistake builds are
    made without OpenMP so that a test process never holds several OpenMP
    thread pools at once."""
    out = out_path or LIB_PATH
    tmp = out + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared",
           "-ffp-contract=off", "-DWBMM_ORACLE_MUTANT=%d" % int(mutant),
           _SRC, "-o", tmp]
    if openmp:
        cmd.insert(1, "-fopenmp")
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def _bind(lib):
    dp = ctypes.POINTER(ctypes.c_double)
    i64 = ctypes.c_int64
    ci = ctypes.c_int
    lib.wbmm_oracle_forward.argtypes = [dp, dp, dp, i64, i64, i64, i64, ci, ci]
    lib.wbmm_oracle_backward_input.argtypes = [dp, dp, dp, i64, i64, i64, i64, ci, ci]
    lib.wbmm_oracle_backward_table.argtypes = [dp, dp, dp, i64, i64, i64, i64, ci, ci]
    lib.wbmm_oracle_relative_index.argtypes = [ci, ci, ctypes.POINTER(ctypes.c_int32)]
    lib.wbmm_oracle_hier_fused_matrix.argtypes = [dp, dp, dp, i64, ci]
    lib.wbmm_oracle_dense_forward.argtypes = [dp, dp, dp, i64, i64, i64, i64, ci, ci]
    lib.wbmm_oracle_dense_backward_matrix.argtypes = [dp, dp, dp, i64, i64, i64, i64, ci, ci]
    lib.wbmm_oracle_set_threads.argtypes = [ci]
    lib.wbmm_oracle_max_threads.restype = ci
    for f in ("wbmm_oracle_forward", "wbmm_oracle_backward_input",
              "wbmm_oracle_backward_table", "wbmm_oracle_relative_index",
              "wbmm_oracle_hier_fused_matrix", "wbmm_oracle_dense_forward",
              "wbmm_oracle_dense_backward_matrix", "wbmm_oracle_set_threads"):
        getattr(lib, f).restype = None
    return lib


def load(path: str | None = None):
    """Load (building first if absent) the oracle shared library."""
    global _lib
    if path is not None:
        return _bind(ctypes.CDLL(path))
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build()
        _lib = _bind(ctypes.CDLL(LIB_PATH))
    return _lib


def _p(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _win(w):
    if isinstance(w, (tuple, list)):
        return int(w[0]), int(w[1])
    return int(w), int(w)


def set_threads(n: int) -> None:
    load().wbmm_oracle_set_threads(int(n))


def max_threads() -> int:
    return int(load().wbmm_oracle_max_threads())


def relative_index(w, lib=None) -> np.ndarray:
    """I[i, j] (eq. index_computation), int32 [d, d]."""
    wh, ww = _win(w)
    d = wh * ww
    out = np.empty((d, d), dtype=np.int32)
    (lib or load()).wbmm_oracle_relative_index(
        wh, ww, out.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)))
    return out


def forward(x, t, w, lib=None) -> np.ndarray:
    """Y = WBMM(X; T, w) in fp64.  x: [B,C,H,W], t: [C,(2wh-1)(2ww-1)]."""
    wh, ww = _win(w)
    x, t = _f64(x), _f64(t)
    B, C, H, W = x.shape
    assert t.shape == (C, (2 * wh - 1) * (2 * ww - 1)), t.shape
    y = np.empty_like(x)
    (lib or load()).wbmm_oracle_forward(_p(x), _p(t), _p(y), B, C, H, W, wh, ww)
    return y


def backward_input(dy, t, w, lib=None) -> np.ndarray:
    """dX of WBMM for upstream gradient dY, fp64."""
    wh, ww = _win(w)
    dy, t = _f64(dy), _f64(t)
    B, C, H, W = dy.shape
    assert t.shape == (C, (2 * wh - 1) * (2 * ww - 1)), t.shape
    dx = np.empty_like(dy)
    (lib or load()).wbmm_oracle_backward_input(_p(dy), _p(t), _p(dx), B, C, H, W, wh, ww)
    return dx


def backward_table(x, dy, w, lib=None) -> np.ndarray:
    """dT of WBMM, fp64 [C, (2wh-1)(2ww-1)]."""
    wh, ww = _win(w)
    x, dy = _f64(x), _f64(dy)
    B, C, H, W = x.shape
    assert dy.shape == x.shape
    dt = np.empty((C, (2 * wh - 1) * (2 * ww - 1)), dtype=np.float64)
    (lib or load()).wbmm_oracle_backward_table(_p(x), _p(dy), _p(dt), B, C, H, W, wh, ww)
    return dt


def hier_fused_matrix(tg, tl, wl, lib=None) -> np.ndarray:
    """M_fused [C, d, d] (d = (2 wl)^2) of the hierarchical reparameterisation."""
    tg, tl = _f64(tg), _f64(tl)
    C = tg.shape[0]
    d = (2 * wl) ** 2
    m = np.empty((C, d, d), dtype=np.float64)
    (lib or load()).wbmm_oracle_hier_fused_matrix(_p(tg), _p(tl), _p(m), C, int(wl))
    return m


def dense_forward(x, m, w, lib=None) -> np.ndarray:
    """Y = X_w M per window with an explicit per-channel matrix M [C, d, d]
    (d = wh ww, positions row-major inside the window; w = wh or (wh, ww))."""
    wh, ww = _win(w)
    x, m = _f64(x), _f64(m)
    B, C, H, W = x.shape
    assert m.shape == (C, wh * ww, wh * ww), m.shape
    y = np.empty_like(x)
    (lib or load()).wbmm_oracle_dense_forward(_p(x), _p(m), _p(y), B, C, H, W, wh, ww)
    return y


def dense_backward_matrix(x, dy, w, lib=None) -> np.ndarray:
    """dM [C, d, d] of the dense form: sum over windows of X_w^T dY_w."""
    wh, ww = _win(w)
    x, dy = _f64(x), _f64(dy)
    B, C, H, W = x.shape
    assert dy.shape == x.shape
    dm = np.empty((C, wh * ww, wh * ww), dtype=np.float64)
    (lib or load()).wbmm_oracle_dense_backward_matrix(_p(x), _p(dy), _p(dm), B, C, H, W, wh, ww)
    return dm


def build_matrix(t, w, lib=None) -> np.ndarray:
    """M_c = R[c, I] (eq. index_select): [C, d, d] from the table [C, K]."""
    wh, ww = _win(w)
    t = _f64(t)
    idx = relative_index((wh, ww), lib=lib).astype(np.int64)
    return np.ascontiguousarray(t[:, idx])


def bin_matrix(dm, w, lib=None) -> np.ndarray:
    """Fold a matrix gradient onto the table: dT[c, k] = sum of dM[c, i, j]
    over the pairs with I[i, j] = k (the adjoint of build_matrix)."""
    wh, ww = _win(w)
    dm = _f64(dm)
    C = dm.shape[0]
    idx = relative_index((wh, ww), lib=lib).astype(np.int64).ravel()
    dt = np.zeros((C, (2 * wh - 1) * (2 * ww - 1)), dtype=np.float64)
    for c in range(C):
        dt[c] = np.bincount(idx, weights=dm[c].ravel(), minlength=dt.shape[1])
    return dt


def hier_forward(x, tg, tl, wl, lib=None) -> np.ndarray:
    """Hierarchical WBMM, inference form: X_w M_fused per global window."""
    return dense_forward(x, hier_fused_matrix(tg, tl, wl, lib=lib), 2 * wl, lib=lib)


def dense_backward_input(dy, m, w, lib=None) -> np.ndarray:
    """dX = dY_w M^T per window for an explicit per-channel matrix M."""
    return dense_forward(dy, np.ascontiguousarray(np.transpose(_f64(m), (0, 2, 1))), w, lib=lib)


def hier_backward_input(dy, tg, tl, wl, lib=None) -> np.ndarray:
    """dX of the hierarchical form: dY_w M_fused^T per global window."""
    return dense_backward_input(dy, hier_fused_matrix(tg, tl, wl, lib=lib), 2 * wl, lib=lib)


def hier_backward_tables(x, dy, wl, lib=None):
    """(dT_g, dT_l) of the hierarchical form.  By the training form
    Y = WBMM(X; T_g, 2 wl) + WBMM(X; T_l, wl) + 2 X (the local sub-windows of
    the zero-padded global windows are the wl windows of the map), each table
    gradient is that of its own scale."""
    return backward_table(x, dy, 2 * wl, lib=lib), backward_table(x, dy, wl, lib=lib)


if __name__ == "__main__":  # pragma: no cover - manual build hook
    print(build(int(sys.argv[1]) if len(sys.argv) > 1 else 0))
