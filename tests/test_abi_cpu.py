"""CPU-side checks of the C-ABI library: it loads, exports every function that
include/wbmm.h declares, and rejects bad arguments on the host before any GPU
work (only argument combinations that fail validation are sent, so no kernel
is ever launched here)."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from paper_2607_02097_amd import binding as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "wbmm.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(wbmm_[a-z_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    return W.load_library()


def test_library_exports_every_declared_function(lib):
    names = declared_functions()
    assert set(names) == set(W.EXPORTED)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings(lib):
    for s in (0, 1, 2, 3, 4):
        assert W.wbmm_status_string(s).startswith("WBMM")
    assert "unknown" in W.wbmm_status_string(77)
    assert W.wbmm_version().count(".") == 2


@pytest.mark.parametrize("w", [1, 2, 5, 7, 14, 16])
def test_relative_index_matches_oracle_bit_exact(lib, w, olib):
    assert np.array_equal(W.wbmm_relative_index(w).numpy(), oracle.relative_index(w, lib=olib))


def test_relative_index_errors(lib):
    buf = (ctypes.c_int32 * 4)()
    assert lib.wbmm_relative_index(0, buf) == W.WBMM_ERR_INVALID_ARG
    assert lib.wbmm_relative_index(17, buf) == W.WBMM_ERR_UNSUPPORTED
    assert lib.wbmm_relative_index(2, None) == W.WBMM_ERR_INVALID_ARG


FAKE = 0x100000  # never dereferenced: every call below fails validation


def fwd(lib, x=FAKE, t=FAKE * 4, y=FAKE * 8, B=1, C=2, H=7, Wd=7, w=7, dt=1, fn="wbmm_forward"):
    return getattr(lib, fn)(ctypes.c_void_p(x), ctypes.c_void_p(t), ctypes.c_void_p(y),
                            B, C, H, Wd, w, dt, None)


@pytest.mark.parametrize("fn", ["wbmm_forward", "wbmm_backward_input"])
def test_forward_like_rejects_bad_arguments(lib, fn):
    E, U = W.WBMM_ERR_INVALID_ARG, W.WBMM_ERR_UNSUPPORTED
    assert fwd(lib, x=0, fn=fn) == E
    assert fwd(lib, t=0, fn=fn) == E
    assert fwd(lib, y=0, fn=fn) == E
    for k in ("B", "C", "H", "Wd"):
        assert fwd(lib, fn=fn, **{k: 0}) == E
        assert fwd(lib, fn=fn, **{k: -3}) == E
    assert fwd(lib, w=0, fn=fn) == E
    assert fwd(lib, w=17, fn=fn) == U
    assert fwd(lib, dt=7, fn=fn) == U
    assert fwd(lib, x=FAKE + 1, fn=fn) == E            # misaligned bf16 pointer
    assert fwd(lib, y=FAKE, fn=fn) == E                # output aliases input
    assert fwd(lib, y=FAKE + 2 * 49, fn=fn) == E      # output overlaps input tail
    assert fwd(lib, B=2 ** 40, C=2 ** 20, fn=fn) == E  # size overflow


def test_backward_table_rejects_bad_arguments(lib):
    E = W.WBMM_ERR_INVALID_ARG
    vp = ctypes.c_void_p

    def call(x=FAKE, dy=FAKE * 8, dt=FAKE * 16, ws=0, wsb=0, B=1, C=2, H=7, Wd=7, w=7, d=1):
        return lib.wbmm_backward_table(vp(x), vp(dy), vp(dt), vp(ws), wsb, B, C, H, Wd, w, d, None)

    assert call(x=0) == E
    assert call(dy=0) == E
    assert call(dt=0) == E
    assert call(dt=FAKE * 16 + 2) == E                 # dtable must be 4-byte aligned
    assert call(dt=FAKE) == E                          # dtable overlaps x
    assert call(w=18) == W.WBMM_ERR_UNSUPPORTED
    # a shape that needs a workspace: missing / too small workspace is rejected
    need = lib.wbmm_backward_table_workspace_bytes(64, 192, 28, 28, 14, 1)
    assert need > 0
    assert call(B=64, C=192, H=28, Wd=28, w=14, x=FAKE, dy=FAKE * 64, dt=FAKE * 128) == E
    assert call(B=64, C=192, H=28, Wd=28, w=14, x=FAKE, dy=FAKE * 64, dt=FAKE * 128,
                ws=FAKE * 256, wsb=need - 4) == E


def test_workspace_query(lib):
    assert lib.wbmm_backward_table_workspace_bytes(0, 1, 1, 1, 7, 1) == 0
    assert lib.wbmm_backward_table_workspace_bytes(1, 8, 28, 28, 7, 0) == 0  # one slab
    n = lib.wbmm_backward_table_workspace_bytes(64, 192, 28, 28, 14, 1)
    assert n > 0 and n % (192 * 729 * 4) == 0  # [slabs, C, (2w-1)^2] float32 partial sums


def test_backward_rejects_bad_arguments(lib):
    E = W.WBMM_ERR_INVALID_ARG
    vp = ctypes.c_void_p

    def call(x=FAKE, dy=FAKE * 8, t=FAKE * 12, dx=FAKE * 16, dt=FAKE * 24, ws=0, wsb=0,
             B=1, C=2, H=7, Wd=7, w=7, d=1):
        return lib.wbmm_backward(vp(x), vp(dy), vp(t), vp(dx), vp(dt), vp(ws), wsb,
                                 B, C, H, Wd, w, d, None)

    for k in ("x", "dy", "t", "dx", "dt"):
        assert call(**{k: 0}) == E, k
    assert call(dx=FAKE * 16 + 1) == E             # misaligned bf16 output
    assert call(dt=FAKE * 24 + 2) == E             # dtable must be 4-byte aligned
    assert call(dx=FAKE) == E                      # dx aliases x
    assert call(dx=FAKE * 8 + 64) == E             # dx overlaps dy
    assert call(dx=FAKE * 12 - 64) == E            # dx overlaps the table
    assert call(dt=FAKE * 12) == E                 # dtable overlaps the table
    assert call(dt=FAKE * 16 + 128) == E           # dtable overlaps dx
    assert call(w=18) == W.WBMM_ERR_UNSUPPORTED
    assert call(d=5) == W.WBMM_ERR_UNSUPPORTED
    need = lib.wbmm_backward_workspace_bytes(64, 192, 28, 28, 14, 1)
    assert need == lib.wbmm_backward_table_workspace_bytes(64, 192, 28, 28, 14, 1) > 0
    big = dict(B=64, C=192, H=28, Wd=28, w=14, x=FAKE, dy=FAKE * 64, t=FAKE * 128,
               dx=FAKE * 192, dt=FAKE * 256)
    assert call(**big) == E                                         # no workspace
    assert call(ws=FAKE * 320, wsb=need - 4, **big) == E            # too small
    assert call(ws=FAKE * 192 + 64, wsb=need, **big) == E           # overlaps dx


def test_hier_rejects_bad_arguments(lib):
    E, U = W.WBMM_ERR_INVALID_ARG, W.WBMM_ERR_UNSUPPORTED
    vp = ctypes.c_void_p

    def fwd_call(x=FAKE, tg=FAKE * 4, tl=FAKE * 6, y=FAKE * 8, B=1, C=2, H=14, Wd=14, wl=7, d=1,
                 fn="wbmm_hier_forward"):
        return getattr(lib, fn)(vp(x), vp(tg), vp(tl), vp(y), B, C, H, Wd, wl, d, None)

    for fn in ("wbmm_hier_forward", "wbmm_hier_backward_input"):
        for k in ("x", "tg", "tl", "y"):
            assert fwd_call(fn=fn, **{k: 0}) == E, (fn, k)
        assert fwd_call(fn=fn, wl=0) == E
        assert fwd_call(fn=fn, wl=9) == U
        assert fwd_call(fn=fn, d=4) == U
        assert fwd_call(fn=fn, y=FAKE) == E            # output aliases input
        assert fwd_call(fn=fn, y=FAKE * 6 + 2) == E    # output overlaps the local table
        assert fwd_call(fn=fn, x=FAKE + 1) == E        # misaligned

    def bwd_call(x=FAKE, dy=FAKE * 8, tg=FAKE * 12, tl=FAKE * 14, dx=FAKE * 16, dtg=FAKE * 20, dtl=FAKE * 24,
                 ws=0, wsb=0, B=1, C=2, H=14, Wd=14, wl=7, d=1):
        return lib.wbmm_hier_backward(vp(x), vp(dy), vp(tg), vp(tl), vp(dx), vp(dtg), vp(dtl), vp(ws), wsb,
                                      B, C, H, Wd, wl, d, None)

    for k in ("x", "dy", "tg", "tl", "dx", "dtg", "dtl"):
        assert bwd_call(**{k: 0}) == E, k
    assert bwd_call(dtl=FAKE * 20 + 64) == E          # the two table gradients overlap
    assert bwd_call(dx=FAKE * 8) == E                 # dx aliases dy
    assert bwd_call(wl=9) == U
    need = lib.wbmm_hier_backward_workspace_bytes(64, 192, 28, 28, 7, 1)
    assert need >= max(lib.wbmm_backward_table_workspace_bytes(64, 192, 28, 28, 14, 1),
                       lib.wbmm_backward_table_workspace_bytes(64, 192, 28, 28, 7, 1)) > 0
    big = dict(B=64, C=192, H=28, Wd=28, x=FAKE, dy=FAKE * 64, tg=FAKE * 128, tl=FAKE * 132,
               dx=FAKE * 192, dtg=FAKE * 256, dtl=FAKE * 260)
    assert bwd_call(**big) == E                                  # no workspace
    assert bwd_call(ws=FAKE * 320, wsb=need - 4, **big) == E     # too small


def test_dense_rejects_bad_arguments(lib):
    E, U = W.WBMM_ERR_INVALID_ARG, W.WBMM_ERR_UNSUPPORTED
    vp = ctypes.c_void_p
    assert lib.wbmm_build_matrix(vp(0), vp(FAKE), 2, 3, 5, 1, None) == E
    assert lib.wbmm_build_matrix(vp(FAKE), vp(0), 2, 3, 5, 1, None) == E
    assert lib.wbmm_build_matrix(vp(FAKE), vp(FAKE), 2, 3, 5, 1, None) == E   # m overlaps the table
    assert lib.wbmm_build_matrix(vp(FAKE), vp(FAKE * 8), 2, 17, 5, 1, None) == U
    assert lib.wbmm_build_matrix(vp(FAKE), vp(FAKE * 8), 2, 0, 5, 1, None) == E
    assert lib.wbmm_build_matrix(vp(FAKE), vp(FAKE * 8), 2, 3, 5, 9, None) == U

    def dcall(fn, a=FAKE, m=FAKE * 8, out=FAKE * 16, B=1, C=2, H=9, Wd=10, wh=3, ww=5, d=1):
        return getattr(lib, fn)(vp(a), vp(m), vp(out), B, C, H, Wd, wh, ww, d, None)

    for fn in ("wbmm_dense_forward", "wbmm_dense_backward_input", "wbmm_dense_backward_matrix"):
        assert dcall(fn, a=0) == E, fn
        assert dcall(fn, m=0) == E, fn
        assert dcall(fn, out=0) == E, fn
        assert dcall(fn, ww=17) == U, fn
        assert dcall(fn, B=0) == E, fn
    assert dcall("wbmm_dense_forward", out=FAKE) == E          # output aliases input
    assert dcall("wbmm_dense_forward", out=FAKE * 8 + 64) == E # output overlaps the matrix
    assert dcall("wbmm_dense_backward_matrix", out=FAKE + 8) == E  # dm overlaps x
    assert lib.wbmm_bin_matrix(vp(FAKE), vp(FAKE + 64), 2, 3, 5, None) == E   # overlap
    assert lib.wbmm_bin_matrix(vp(0), vp(FAKE * 8), 2, 3, 5, None) == E
    assert lib.wbmm_bin_matrix(vp(FAKE), vp(FAKE * 8), 2, 3, 0, None) == E


def test_build_rejects_flat_memory_instructions():
    """The build's guard finds flat-address-space accesses in a disassembly
    and names their kernel; ds_*, global_* and buffer_* accesses pass."""
    from paper_2607_02097_amd import build as B
    listing = "\n".join([
        "0000000000001000 <_ZN4wbmm6kernelILi1EEEvv>:",
        "\tds_read_b128 v[0:3], v4",
        "\tglobal_load_dwordx4 v[0:3], v[4:5], off",
        "\tbuffer_load_dword v1, off, s[0:3], 0",
        "0000000000002000 <_ZN4wbmm6kernelILi2EEEvv>:",
        "\tflat_load_dwordx4 v[0:3], v[4:5]",
        "\tflat_store_dword v[4:5], v1",
    ])
    found = B.flat_accesses(listing)
    assert found == [("_ZN4wbmm6kernelILi2EEEvv", "flat_load_dwordx4"),
                     ("_ZN4wbmm6kernelILi2EEEvv", "flat_store_dword")]
    assert B.flat_accesses(listing.split("0000000000002000")[0]) == []


def test_noalloc_validates_on_the_host(lib):
    """wbmm_backward_noalloc rejects bad arguments, and shapes whose scratch
    exceeds the static buffer, before any GPU work (no kernel launch here)."""
    vp = ctypes.c_void_p
    G = 1 << 32  # far-apart fake device addresses: the tensors do not overlap

    def call(x=G, dy=2 * G, t=3 * G, dx=4 * G, dt=5 * G, B=33, C=700, H=16, Wd=16, w=16, d=1):
        return lib.wbmm_backward_noalloc(vp(x), vp(dy), vp(t), vp(dx), vp(dt), B, C, H, Wd, w, d, None)

    need = lib.wbmm_backward_workspace_bytes(33, 700, 16, 16, 16, 1)
    assert need > W.NOALLOC_SCRATCH_BYTES
    assert call() == W.WBMM_ERR_SCRATCH
    assert call(x=0) == W.WBMM_ERR_INVALID_ARG
    assert call(dx=G) == W.WBMM_ERR_INVALID_ARG  # dx aliases x
    assert call(w=17) == W.WBMM_ERR_UNSUPPORTED
    assert "scratch" in W.wbmm_status_string(W.WBMM_ERR_SCRATCH)


def test_float_quotient_without_correction():
    """The image-layout kernels split chunk and lane indices by a divisor d
    with trunc((v + 1/2) * fl(1/d)) in float32 and no correction step; that
    is the integer quotient for 0 <= v < 2^22.  Checked exhaustively with
    IEEE float32 arithmetic (the device's round-to-nearest-even): every d up
    to 4096 with v below 2^13 (chunk, lane and band indices), and every v
    below 2^22 for d up to 48."""
    f = np.float32

    def quotient(v, d):
        return ((v.astype(np.float32) + f(0.5)) * (f(1.0) / f(d))).astype(np.int64)

    v = np.arange(1 << 13, dtype=np.int64)
    for d in range(1, 4097):
        assert np.array_equal(quotient(v, d), v // d), d
    v = np.arange(1 << 22, dtype=np.int64)
    for d in range(1, 49):
        assert np.array_equal(quotient(v, d), v // d), d
