"""The allocation-free backward entry point (wbmm_backward_noalloc, for
callers that cannot allocate device memory) against wbmm_backward: the same
kernels with the table-gradient scratch in the library's static buffer
instead of a caller workspace, so the results must be equal bit for bit.
Two calls in a row share the static buffer, the second with a smaller input;
a shape whose scratch exceeds the buffer is rejected before any GPU work."""
import ctypes

import numpy as np
import pytest
import torch

from helpers import draw, to_device
from paper_2607_02097_amd import binding as W
from paper_2607_02097_amd import synth

pytestmark = pytest.mark.gpu


def noalloc_via_abi(x, dy, t, w, dx, dt):
    """One call through the C ABI on torch's current stream."""
    lib = W.load_library()
    vp = ctypes.c_void_p
    B, C, H, Wd = x.shape
    st = vp(torch.cuda.current_stream().cuda_stream)
    return lib.wbmm_backward_noalloc(vp(x.data_ptr()), vp(dy.data_ptr()), vp(t.data_ptr()), vp(dx.data_ptr()),
                                     vp(dt.data_ptr()), B, C, H, Wd, w, W.DTYPE_CODES[x.dtype], st)


def compare(d, w, dtype, label):
    x, t, dy = (to_device(d[k], dtype) for k in ("x", "t", "dy"))
    ref_dx, ref_dt = W.wbmm_backward(x, dy, t, w)
    dx = torch.full_like(x, float("nan"))
    dt = torch.full_like(ref_dt, float("nan"))
    r = noalloc_via_abi(x, dy, t, w, dx, dt)
    torch.cuda.synchronize()
    assert r == W.WBMM_OK, "%s: %s" % (label, W.wbmm_status_string(r))
    assert torch.equal(dx, ref_dx), "%s: dx differs from wbmm_backward" % label
    assert torch.equal(dt, ref_dt), "%s: dtable differs from wbmm_backward" % label
    need = W.wbmm_backward_workspace_bytes(x.shape, w, x.dtype)
    print("[noalloc] %s scratch %d bytes: equal" % (label, need), flush=True)
    return need


def test_noalloc_two_calls_then_smaller():
    """Two calls in a row on the static scratch, the second with a smaller
    input (fewer channels and windows), each equal to wbmm_backward bit for
    bit; both shapes use the scratch (several slabs per channel)."""
    big = synth.WORKLOADS["bf16_b16_c64_112_w14"]
    d = synth.draw_workload(big, seed=3)
    n1 = compare(d, 14, "bf16", "B16 C64 112 w14")
    d2 = draw(4, 24, 112, 112, 14, "bf16", seed=4)
    n2 = compare(d2, 14, "bf16", "B4 C24 112 w14")
    assert n1 > 0 and n2 > 0


@pytest.mark.parametrize("shape,dtype", [
    ((128, 384, 14, 14, 14), "bf16"),  # more channels than compute units: four-wave kernels, 3 slabs
    ((6, 3, 30, 17, 14), "f32"),       # ragged map: generic rows, 3 slabs
    ((5, 3, 56, 56, 7), "f16"),
])
def test_noalloc_matches_workspace_entry_point(shape, dtype):
    B, C, H, Wd, w = shape
    compare(draw(B, C, H, Wd, w, dtype, seed=9), w, dtype, "%s %s" % (dtype, shape))


def test_noalloc_rejects_oversized_scratch():
    """A shape whose table-gradient scratch exceeds the static buffer is
    refused with WBMM_ERR_SCRATCH, and the outputs stay untouched."""
    B, C, H, Wd, w = 33, 700, 16, 16, 16
    need = W.wbmm_backward_workspace_bytes((B, C, H, Wd), w, torch.bfloat16)
    assert need > W.NOALLOC_SCRATCH_BYTES
    x = torch.zeros((B, C, H, Wd), dtype=torch.bfloat16, device="cuda")
    dy = torch.zeros_like(x)
    t = torch.zeros((C, (2 * w - 1) ** 2), dtype=torch.bfloat16, device="cuda")
    dx = torch.full_like(x, 7.0)
    dt = torch.full((C, (2 * w - 1) ** 2), 7.0, dtype=torch.float32, device="cuda")
    assert noalloc_via_abi(x, dy, t, w, dx, dt) == W.WBMM_ERR_SCRATCH
    torch.cuda.synchronize()
    assert bool((dx == 7.0).all()) and bool((dt == 7.0).all())
