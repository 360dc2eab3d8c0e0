"""GPU parity: the HIP path (through the C ABI) against the fp64 CPU oracle.

* small shapes spanning several workgroup tiles, ragged tails and padding, for
  every dtype, at the stated tolerances (infinity-norm relative error);
* bit-exact checks of the window/index mapping: one-hot tables (each output is
  one input value or 0) and small-integer data (every sum exact);
* every window size 1..16;
* the five workloads at full size, in the launch configuration the benchmark
  uses, against the oracle on every channel;
* more channels than the device has compute units (the four-wave gradient
  kernels, the channel stream in rounds and in runs of stages), in every
  dtype, with an exact small-integer variant;
* a seeded sweep of random shapes over every pass and the fused backward;
* determinism, non-default streams, the autograd composition, error paths.
"""
import numpy as np
import pytest
import torch

import oracle
from helpers import TOL, TORCH_DTYPE, draw, rel_inf, to_device, to_f64, tol_for
from paper_2607_02097_amd import binding as W
from paper_2607_02097_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu_ready():
    assert torch.cuda.is_available(), "the GPU tests need a ROCm GPU"
    W.load_library()
    print("\n[gpu] device:", torch.cuda.get_device_name(0), flush=True)


def run_gpu(d, w, dtype, passes=("fwd", "dx", "dt")):
    x = to_device(d["x"], dtype)
    t = to_device(d["t"], dtype)
    dy = to_device(d["dy"], dtype)
    out = {}
    if "fwd" in passes:
        out["fwd"] = W.wbmm_forward(x, t, w)
    if "dx" in passes:
        out["dx"] = W.wbmm_backward_input(dy, t, w)
    if "dt" in passes:
        out["dt"] = W.wbmm_backward_table(x, dy, w)
    torch.cuda.synchronize()
    return {k: to_f64(v) for k, v in out.items()}


def run_oracle(d, w, passes=("fwd", "dx", "dt")):
    out = {}
    if "fwd" in passes:
        out["fwd"] = oracle.forward(d["x64"], d["t64"], w)
    if "dx" in passes:
        out["dx"] = oracle.backward_input(d["dy64"], d["t64"], w)
    if "dt" in passes:
        out["dt"] = oracle.backward_table(d["x64"], d["dy64"], w)
    return out


def check(got, want, dtype, label):
    for k in want:
        assert np.isfinite(got[k]).all(), "%s %s: non-finite output" % (label, k)
        e = rel_inf(got[k], want[k])
        tol = tol_for(k, dtype)
        print("[parity] %s %s rel_err=%.3e (tol %.0e)" % (label, k, e, tol), flush=True)
        assert e <= tol, "%s %s: rel err %.3e > %.1e" % (label, k, e, tol)


SMALL = [
    # (B, C, H, W, w): several tiles, ragged tails, padding on either axis
    (1, 8, 28, 28, 7),
    (3, 5, 21, 35, 7),
    (5, 3, 56, 56, 7),
    (2, 2, 10, 13, 7),
    (3, 4, 28, 42, 14),
    (20, 3, 28, 28, 14),
    (2, 3, 30, 17, 14),
    (1, 2, 14, 14, 14),
    (9, 2, 14, 14, 14),
    # wide images: many windows per band, ragged bottom windows
    (1, 2, 20, 600, 14),
    (2, 1, 9, 1200, 7),
]


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("shape", SMALL, ids=lambda s: "B%dC%dH%dW%dw%d" % s)
def test_small_parity(shape, dtype):
    B, C, H, Wd, w = shape
    d = draw(B, C, H, Wd, w, dtype, seed=11)
    check(run_gpu(d, w, dtype), run_oracle(d, w), dtype, "%s %s" % (dtype, shape))


def check_fused(d, w, dtype, label):
    """The fused backward equals the two separate entry points bit for bit
    (same products, same summation orders) and the oracle within tolerance."""
    x, t, dy = (to_device(d[k], dtype) for k in ("x", "t", "dy"))
    dx, dt = W.wbmm_backward(x, dy, t, w)
    dx_s = W.wbmm_backward_input(dy, t, w)
    dt_s = W.wbmm_backward_table(x, dy, w)
    torch.cuda.synchronize()
    assert torch.equal(dx, dx_s), "%s: fused dx differs from wbmm_backward_input" % label
    assert torch.equal(dt, dt_s), "%s: fused dt differs from wbmm_backward_table" % label
    check({"dx": to_f64(dx), "dt": to_f64(dt)}, run_oracle(d, w, ("dx", "dt")), dtype, label + " fused")


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("shape", SMALL, ids=lambda s: "B%dC%dH%dW%dw%d" % s)
def test_fused_backward_small(shape, dtype):
    B, C, H, Wd, w = shape
    d = draw(B, C, H, Wd, w, dtype, seed=12)
    check_fused(d, w, dtype, "%s %s" % (dtype, shape))


# shapes whose gradient kernels take fixed-offset rows (windows tile the map,
# NW a power of two, 16-window sub-tiles are whole bands of one image or whole
# images; 16-bit needs an even window)
TILED = [
    (20, 3, 28, 28, 14),   # four images per sub-tile
    (3, 2, 28, 28, 14),    # a partial sub-tile (three images)
    (9, 2, 14, 14, 14),    # one window per image, partial sub-tile
    (1, 2, 112, 112, 14),  # bands of one image
    (2, 2, 32, 64, 16),
    (4, 3, 24, 24, 12),
    (2, 3, 40, 40, 10),
    (3, 2, 18, 36, 9),     # odd window: float32 only
    (5, 3, 56, 56, 7),     # odd window: float32 only
]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", TILED, ids=lambda s: "B%dC%dH%dW%dw%d" % s)
def test_fixed_offset_rows_backward(shape, dtype):
    """Forward and gradients on tensors whose rows the kernels address by
    fixed offsets equal those on misaligned copies (generic row addressing)
    bit for bit, and the oracle within tolerance."""
    B, C, H, Wd, w = shape
    d = draw(B, C, H, Wd, w, dtype, seed=31)
    x, t, dy = (to_device(d[k], dtype) for k in ("x", "t", "dy"))
    dx, dt = W.wbmm_backward(x, dy, t, w)
    dt_s = W.wbmm_backward_table(x, dy, w)
    y = W.wbmm_forward(x, t, w)
    if dtype != "f32":
        xm, dym = misaligned_like(x), misaligned_like(dy)
        dxm = misaligned_like(torch.zeros_like(dy))
        ym = misaligned_like(torch.zeros_like(x))
        dtm = torch.empty_like(dt)
        W.wbmm_backward(xm, dym, t, w, dx=dxm, dtable=dtm)
        dtm2 = W.wbmm_backward_table(xm, dym, w)
        W.wbmm_forward(xm, t, w, out=ym)
        torch.cuda.synchronize()
        assert torch.equal(dx, dxm) and torch.equal(y, ym)
        # few channels per compute unit: the fixed-offset gradients stream
        # each channel through one workgroup, the generic kernels split it into
        # slabs; the same products summed in another order
        assert torch.equal(dtm, dtm2)
        scale = float(dt.abs().max()) + 1e-30
        assert float((dt - dtm).abs().max()) <= 1e-5 * scale
    torch.cuda.synchronize()
    assert torch.equal(dt, dt_s)
    check({"fwd": to_f64(y), "dx": to_f64(dx), "dt": to_f64(dt)}, run_oracle(d, w, ("fwd", "dx", "dt")), dtype,
          "tiled %s %s" % (dtype, shape))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("w", list(range(1, 17)))
def test_fused_backward_every_window_size(w, dtype):
    B, C, H, Wd = 3, 2, 2 * w + 3, w + 5
    d = draw(B, C, H, Wd, w, dtype, seed=100 + w)
    check_fused(d, w, dtype, "%s w=%d" % (dtype, w))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("w", list(range(1, 17)))
def test_every_window_size(w, dtype):
    B, C, H, Wd = 3, 2, 2 * w + 3, w + 5
    d = draw(B, C, H, Wd, w, dtype, seed=w)
    check(run_gpu(d, w, dtype), run_oracle(d, w), dtype, "%s w=%d" % (dtype, w))


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("w", [7, 14])
def test_one_hot_table_bit_exact(w, dtype):
    """T[c] = e_k: each output is exactly one input value or zero, so the GPU
    result must equal the oracle bit for bit (window and index mapping)."""
    B, C, H, Wd = 3, 6, 2 * w + 3, 3 * w - 2
    d = draw(B, C, H, Wd, w, dtype, seed=5)
    K = 2 * w - 1
    t64 = np.zeros((C, K * K))
    offs = [(0, 0), (1, -2), (-(w - 1), w - 1), (w - 1, -(w - 1)), (-3, 0), (2, 5)]
    for c in range(C):
        dh, dw = offs[c]
        t64[c, (dh + w - 1) * K + (dw + w - 1)] = 1.0
    d["t"], d["t64"] = synth.round_to(t64, dtype)
    got = run_gpu(d, w, dtype, ("fwd", "dx"))
    want = run_oracle(d, w, ("fwd", "dx"))
    for k in want:
        assert np.array_equal(got[k], want[k]), k


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("w", [7, 14])
def test_integer_data_bit_exact(w, dtype):
    """Small integers: every product and partial sum is exact in fp32 and every
    output is an integer below 256 in magnitude, exactly representable in the
    16-bit types, so all three results must match the oracle exactly."""
    B, C, H, Wd = 4, 3, 3 * w - 1, 2 * w
    r = np.random.default_rng(9)
    lim = 2 if w == 7 else 1
    x64 = r.integers(-lim, lim + 1, size=(B, C, H, Wd)).astype(np.float64)
    dy64 = r.integers(-lim, lim + 1, size=(B, C, H, Wd)).astype(np.float64)
    t64 = r.integers(-lim, lim + 1, size=(C, (2 * w - 1) ** 2)).astype(np.float64)
    d = {}
    for k, a in (("x", x64), ("t", t64), ("dy", dy64)):
        d[k], d[k + "64"] = synth.round_to(a, dtype)
    got = run_gpu(d, w, dtype)
    want = run_oracle(d, w)
    for k in want:
        assert np.array_equal(got[k], want[k]), k


# maps the windows tile, few channels: the channel-stream gradients (one
# workgroup per channel, or several slabs with a ticket) and the image-layout
# forward
TILED_EXACT = [
    (16, 3, 28, 28, 14),   # one slab per channel
    (2, 2, 112, 112, 14),  # four slabs per channel, parts summed by ticket
    (8, 2, 40, 40, 10),
    (4, 3, 32, 64, 16),
]


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("shape", TILED_EXACT, ids=lambda s: "B%dC%dH%dW%dw%d" % s)
def test_fixed_offset_integer_data_bit_exact(shape, dtype):
    """Integers in {-1, 0, 1} on maps the windows tile: every sum is exact in
    fp32 and every output an integer below 256, so the forward, both
    gradients and the fused backward must equal the oracle bit for bit."""
    B, C, H, Wd, w = shape
    r = np.random.default_rng(11 + w)
    d = {}
    for k, shp in (("x", (B, C, H, Wd)), ("dy", (B, C, H, Wd)), ("t", (C, (2 * w - 1) ** 2))):
        d[k], d[k + "64"] = synth.round_to(r.integers(-1, 2, size=shp).astype(np.float64), dtype)
    got = run_gpu(d, w, dtype)
    x, t, dy = (to_device(d[k], dtype) for k in ("x", "t", "dy"))
    dx, dt = W.wbmm_backward(x, dy, t, w)
    torch.cuda.synchronize()
    got["fused dx"], got["fused dt"] = to_f64(dx), to_f64(dt)
    want = run_oracle(d, w)
    want["fused dx"], want["fused dt"] = want["dx"], want["dt"]
    for k in want:
        assert np.array_equal(got[k], want[k]), k


# shapes for the image-layout forward (16-bit, windows tile the map, NW a
# power of two, a 16-window sub-tile is whole bands of one image or whole
# images, pieces 16-byte aligned)
IMG = [
    (5, 3, 56, 56, 7),
    (3, 2, 14, 56, 7),     # 16 windows per image; ragged last tile
    (2, 3, 16, 16, 4),     # 4 windows per band
    (1, 2, 24, 64, 8),     # 24 windows per image: neither layout, row path
    (2, 2, 8, 32, 2),      # 16 windows per band
    (3, 2, 5, 40, 5),      # one band per image, two images per sub-tile, partial last sub-tile
    (1, 4, 16, 16, 1),
    (4, 3, 28, 28, 14),    # four images per sub-tile
    (3, 2, 28, 28, 14),    # three images in the only sub-tile
    (1, 2, 112, 112, 14),  # bands of one image
    (2, 3, 24, 48, 12),
    (5, 2, 16, 32, 16),    # eight images per sub-tile, partial
    (2, 2, 18, 36, 9),     # odd window (2-byte result writes), rows stored per sub-tile
    (1, 2, 30, 60, 15),
]


def misaligned_like(t):
    """A contiguous copy of t whose data starts 2 bytes past a 16-byte boundary
    (the forward then takes the row path)."""
    buf = torch.empty(t.numel() + 8, dtype=t.dtype, device=t.device)
    v = buf[1:1 + t.numel()].view(t.shape)
    v.copy_(t)
    return v


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("shape", IMG, ids=lambda s: "B%dC%dH%dW%dw%d" % s)
def test_image_layout_forward(shape, dtype):
    """The image-layout forward and input gradient match the oracle and equal
    the row-path results bit for bit (same products, same order)."""
    B, C, H, Wd, w = shape
    d = draw(B, C, H, Wd, w, dtype, seed=21)
    x, t, dy = (to_device(d[k], dtype) for k in ("x", "t", "dy"))
    y, dx = W.wbmm_forward(x, t, w), W.wbmm_backward_input(dy, t, w)
    xm, dym = misaligned_like(x), misaligned_like(dy)
    ym, dxm = misaligned_like(torch.zeros_like(x)), misaligned_like(torch.zeros_like(dy))
    W.wbmm_forward(xm, t, w, out=ym)
    W.wbmm_backward_input(dym, t, w, out=dxm)
    torch.cuda.synchronize()
    assert torch.equal(y, ym) and torch.equal(dx, dxm)
    check({"fwd": to_f64(y), "dx": to_f64(dx)}, run_oracle(d, w, ("fwd", "dx")), dtype, "image layout %s" % (shape,))


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("w", [7, 14])
def test_image_layout_one_hot_bit_exact(dtype, w):
    B, C, H, Wd = (2, 6, 14, 56) if w == 7 else (3, 6, 28, 28)
    d = draw(B, C, H, Wd, w, dtype, seed=6)
    K = 2 * w - 1
    t64 = np.zeros((C, K * K))
    offs = [(0, 0), (1, -2), (-(w - 1), w - 1), (w - 1, -(w - 1)), (-3, 0), (2, 5)]
    for c in range(C):
        dh, dw = offs[c]
        t64[c, (dh + w - 1) * K + (dw + w - 1)] = 1.0
    d["t"], d["t64"] = synth.round_to(t64, dtype)
    got = run_gpu(d, w, dtype, ("fwd", "dx"))
    want = run_oracle(d, w, ("fwd", "dx"))
    for k in want:
        assert np.array_equal(got[k], want[k]), k


@pytest.mark.parametrize("name", list(synth.WORKLOADS))
def test_workload_full_size(name):
    """Full-size run in the benchmark's launch configuration against the
    oracle on every channel and window."""
    wl = synth.WORKLOADS[name]
    d = synth.draw_workload(wl, seed=0)
    print("[workload] %s passes=%s" % (name, ",".join(wl.passes)), flush=True)
    got = run_gpu(d, wl.w, wl.dtype, wl.passes)
    for k, v in got.items():
        assert np.isfinite(v).all(), "%s %s: non-finite output" % (name, k)
    check(got, run_oracle(d, wl.w, wl.passes), wl.dtype, name)
    if "dt" in wl.passes:
        # the fused backward at full size: equal to the separate passes
        x, t, dy = (to_device(d[k], wl.dtype) for k in ("x", "t", "dy"))
        dx, dt = W.wbmm_backward(x, dy, t, wl.w)
        torch.cuda.synchronize()
        assert np.array_equal(to_f64(dx), got["dx"]), "%s: fused dx" % name
        assert np.array_equal(to_f64(dt), got["dt"]), "%s: fused dt" % name


# more channels than compute units: the gradients take the four-wave kernels
# (fixed-offset rows where the map allows them: f32 at every window, 16-bit
# at even windows), one workgroup per (channel, slab)
MANY_CH = [
    (2, 260, 28, 28, 14),  # four images per sub-tile
    (3, 260, 14, 14, 14),  # one window per image
    (1, 260, 28, 28, 7),   # sixteen windows per image (bands); 16-bit: generic rows
    (2, 259, 21, 30, 7),   # ragged and padded: generic rows
]


def compute_units():
    return torch.cuda.get_device_properties(0).multi_processor_count


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("shape", MANY_CH, ids=lambda s: "B%dC%dH%dW%dw%d" % s)
def test_more_channels_than_compute_units(shape, dtype):
    B, C, H, Wd, w = shape
    assert C > compute_units(), "the shape must have more channels than the device's compute units"
    d = draw(B, C, H, Wd, w, dtype, seed=61)
    check_fused(d, w, dtype, "channels>CUs %s %s" % (dtype, shape))
    y = W.wbmm_forward(to_device(d["x"], dtype), to_device(d["t"], dtype), w)
    torch.cuda.synchronize()
    check({"fwd": to_f64(y)}, run_oracle(d, w, ("fwd",)), dtype, "channels>CUs %s %s" % (dtype, shape))


# more channels than compute units with a last round at least half full: the
# gradients stream whole channels in two rounds of one workgroup per compute
# unit (fused and separate alike)
TWO_ROUNDS = [
    (2, 384, 28, 28, 14),  # 384 = 256 + 128 on 256 compute units
    (1, 400, 28, 56, 14),  # 400 = 256 + 144; eight windows per image
]


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("shape", TWO_ROUNDS, ids=lambda s: "B%dC%dH%dW%dw%d" % s)
def test_channel_stream_in_rounds(shape, dtype):
    B, C, H, Wd, w = shape
    ncu = compute_units()
    assert C > ncu and C % ncu >= ncu // 2
    d = draw(B, C, H, Wd, w, dtype, seed=61)
    check_fused(d, w, dtype, "rounds %s %s" % (dtype, shape))


# more channels than compute units with at least two stages per channel
# (16-bit): runs of consecutive stages over all channels, one workgroup per
# compute unit; a channel is split between two runs (two partial tables, added
# by the sum kernel) or lies whole in one (its second partial zero).  Float32
# takes the other paths and is checked the same way.
RUNS = [
    (64, 300, 14, 14, 14),  # 2 stages per channel, runs of 3
    (32, 288, 28, 28, 14),  # 4 stages per channel, runs of 5
]


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("shape", RUNS, ids=lambda s: "B%dC%dH%dW%dw%d" % s)
def test_channel_stream_runs(shape, dtype):
    B, C, H, Wd, w = shape
    assert C > compute_units()
    d = draw(B, C, H, Wd, w, dtype, seed=67)
    check_fused(d, w, dtype, "runs %s %s" % (dtype, shape))


@pytest.mark.parametrize("shape", RUNS, ids=lambda s: "B%dC%dH%dW%dw%d" % s)
def test_channel_stream_runs_workspace_contents_do_not_matter(shape):
    """The runs' partial tables (both slots of every channel, the zero second
    slot of a channel whole in one run) are written before they are read: a
    workspace holding NaN on entry gives the result of a fresh one."""
    B, C, H, Wd, w = shape
    d = draw(B, C, H, Wd, w, "bf16", seed=69)
    x, dy, t = (to_device(d[k], "bf16") for k in ("x", "dy", "t"))
    need = W.wbmm_backward_table_workspace_bytes(x.shape, w, x.dtype)
    assert need >= 2 * C * (2 * w - 1) ** 2 * 4
    ref = W.wbmm_backward_table(x, dy, w, workspace=W.new_workspace(need))
    ws = garbage_workspace(need)
    got = W.wbmm_backward_table(x, dy, w, workspace=ws)
    _, got2 = W.wbmm_backward(x, dy, t, w, workspace=garbage_workspace(need))
    torch.cuda.synchronize()
    assert torch.equal(got, ref) and torch.equal(got2, ref)


def check_integer_exact(shape, dtype, seed):
    """Integers in {-1, 0, 1}: every sum is exact, so the forward and both
    gradients (separate and fused) equal the oracle bit for bit."""
    B, C, H, Wd, w = shape
    r = np.random.default_rng(seed)
    d = {}
    for k, shp in (("x", (B, C, H, Wd)), ("dy", (B, C, H, Wd)), ("t", (C, (2 * w - 1) ** 2))):
        d[k], d[k + "64"] = synth.round_to(r.integers(-1, 2, size=shp).astype(np.float64), dtype)
    got = run_gpu(d, w, dtype)
    x, t, dy = (to_device(d[k], dtype) for k in ("x", "t", "dy"))
    dx, dt = W.wbmm_backward(x, dy, t, w)
    torch.cuda.synchronize()
    got["fused dx"], got["fused dt"] = to_f64(dx), to_f64(dt)
    want = run_oracle(d, w)
    want["fused dx"], want["fused dt"] = want["dx"], want["dt"]
    for k in want:
        assert np.array_equal(got[k], want[k]), k


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("shape", MANY_CH, ids=lambda s: "B%dC%dH%dW%dw%d" % s)
def test_more_channels_integer_data_bit_exact(shape, dtype):
    assert shape[1] > compute_units()
    check_integer_exact(shape, dtype, 71 + shape[4])


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("shape", RUNS, ids=lambda s: "B%dC%dH%dW%dw%d" % s)
def test_channel_stream_runs_integer_bit_exact(shape, dtype):
    assert shape[1] > compute_units()
    check_integer_exact(shape, dtype, 101 + shape[1])


# few stages per channel and fewer channels than compute units: the fused
# gradients split each channel's windows into slabs of one or two stages
# each, so most slabs are short and the last one is ragged
SHORT_SLABS = [
    (40, 60, 28, 28, 14),  # 16-bit: 5 stages per channel in slabs of 2, 2, 1; float32: 10 in 3, 3, 3, 1
    (24, 90, 24, 24, 12),  # 16-bit: 3 stages per channel in slabs of 2, 1; float32: 6 in 3, 3
]


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("shape", SHORT_SLABS, ids=lambda s: "B%dC%dH%dW%dw%d" % s)
def test_short_slabs(shape, dtype):
    B, C, H, Wd, w = shape
    d = draw(B, C, H, Wd, w, dtype, seed=81)
    check_fused(d, w, dtype, "short slabs %s %s" % (dtype, shape))


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("shape", TWO_ROUNDS, ids=lambda s: "B%dC%dH%dW%dw%d" % s)
def test_channel_stream_in_rounds_integer_bit_exact(shape, dtype):
    check_integer_exact(shape, dtype, 97 + shape[1])


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("shape", SHORT_SLABS, ids=lambda s: "B%dC%dH%dW%dw%d" % s)
def test_short_slabs_integer_bit_exact(shape, dtype):
    check_integer_exact(shape, dtype, 91 + shape[4])


def test_determinism_and_reversed_table():
    wl = synth.WORKLOADS["bf16_b64_c192_28_w14"]
    d = synth.draw_workload(wl, seed=1)
    x, t, dy = (to_device(d[k], "bf16") for k in ("x", "t", "dy"))
    a = [W.wbmm_backward_table(x, dy, 14) for _ in range(2)]
    f = [W.wbmm_forward(x, t, 14) for _ in range(2)]
    dx = W.wbmm_backward_input(dy, t, 14)
    rev = W.wbmm_forward(dy, t.flip(1).contiguous(), 14)
    torch.cuda.synchronize()
    assert torch.equal(a[0], a[1])
    assert torch.equal(f[0], f[1])
    assert torch.equal(dx, rev)  # M^T is the matrix of the reversed table


def test_nondefault_stream():
    d = draw(4, 3, 28, 28, 14, "bf16", seed=3)
    x, t, dy = (to_device(d[k], "bf16") for k in ("x", "t", "dy"))
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        y = W.wbmm_forward(x, t, 14)
        g = W.wbmm_backward_table(x, dy, 14)
    s.synchronize()
    check({"fwd": to_f64(y), "dt": to_f64(g)}, run_oracle(d, 14, ("fwd", "dt")), "bf16", "stream")


def test_cached_workspace_on_explicit_stream():
    """A call on a stream that is not the current one, with the binding's own
    cached workspace created for it (on that stream), while the current
    stream is still busy."""
    B, C, H, Wd, w = 3, 2, 112, 112, 14  # several slabs per channel: workspace in use
    d = draw(B, C, H, Wd, w, "bf16", seed=8)
    x, dy = (to_device(d[k], "bf16") for k in ("x", "dy"))
    assert W.wbmm_backward_table_workspace_bytes(x.shape, w, x.dtype) > 0
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    busy = torch.ones(4096, 4096, device="cuda")
    for _ in range(8):
        busy = busy @ busy * (1.0 / 4096)  # keeps the current stream busy
    g = W.wbmm_backward_table(x, dy, w, stream=s)
    s.synchronize()
    torch.cuda.synchronize()
    check({"dt": to_f64(g)}, run_oracle(d, w, ("dt",)), "bf16", "explicit stream")


def test_autograd_function():
    d = draw(2, 3, 14, 21, 7, "f32", seed=4)
    x = to_device(d["x"], "f32").requires_grad_(True)
    t = to_device(d["t"], "f32").requires_grad_(True)
    dy = to_device(d["dy"], "f32")
    y = W.wbmm(x, t, 7)
    y.backward(dy)
    torch.cuda.synchronize()
    want = run_oracle(d, 7)
    check({"fwd": to_f64(y), "dx": to_f64(x.grad), "dt": to_f64(t.grad)}, want, "f32", "autograd")


def test_gpu_error_paths():
    x = torch.zeros((1, 2, 7, 7), dtype=torch.bfloat16, device="cuda")
    t = torch.zeros((2, 169), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(W.WbmmError):
        W.wbmm_forward(x, t, 17)
    with pytest.raises(ValueError):
        W.wbmm_forward(x, t.float(), 7)
    with pytest.raises(W.WbmmError):
        W.wbmm_forward(x, t, 7, out=x)  # output aliases the input
    big = torch.zeros((64, 192, 28, 28), dtype=torch.bfloat16, device="cuda")
    need = W.wbmm_backward_table_workspace_bytes(big.shape, 14, big.dtype)
    ws = W.new_workspace(need - 4)
    with pytest.raises(W.WbmmError):
        W.wbmm_backward_table(big, big.clone(), 14, workspace=ws)
    tb = torch.zeros((192, 729), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(W.WbmmError):
        W.wbmm_backward(big, big.clone(), tb, 14, workspace=ws)  # workspace too small
    with pytest.raises(W.WbmmError):
        W.wbmm_backward(x, x.clone(), t, 7, dx=x)  # dx aliases x


def test_hip_graph_replay_matches_eager():
    """The three entry points allocate nothing and record no memset, so they
    can be captured in a HIP graph; every replay (with eager work and
    synchronisations in between) must reproduce the eager results exactly."""
    wl = synth.WORKLOADS["bf16_b64_c192_28_w14"]
    d = synth.draw_workload(wl, seed=2)
    x, t, dy = (to_device(d[k], "bf16") for k in ("x", "t", "dy"))
    need = W.wbmm_backward_table_workspace_bytes(x.shape, 14, x.dtype)
    ws = W.new_workspace(need)
    y, dx, dx2 = torch.empty_like(x), torch.empty_like(dy), torch.empty_like(dy)
    dt = torch.empty((wl.C, wl.table_len), dtype=torch.float32, device="cuda")
    dt2 = torch.empty_like(dt)
    ref = (W.wbmm_forward(x, t, 14), W.wbmm_backward_input(dy, t, 14),
           W.wbmm_backward_table(x, dy, 14, workspace=ws))
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.graph(g, stream=s):
        W.wbmm_forward(x, t, 14, out=y)
        W.wbmm_backward_input(dy, t, 14, out=dx)
        W.wbmm_backward_table(x, dy, 14, out=dt, workspace=ws)
        W.wbmm_backward(x, dy, t, 14, dx=dx2, dtable=dt2, workspace=ws)
    torch.cuda.current_stream().wait_stream(s)
    for rep in range(3):
        y.zero_(); dx.zero_(); dt.zero_(); dx2.zero_(); dt2.zero_()
        W.wbmm_forward(dy, t, 14)  # unrelated eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, ref[0]) and torch.equal(dx, ref[1]) and torch.equal(dt, ref[2]), rep
        assert torch.equal(dx2, ref[1]) and torch.equal(dt2, ref[2]), rep


def garbage_workspace(nbytes):
    """A workspace filled with 0xff bytes (NaN as float32): the library must
    not read anything it has not written in the same call."""
    return torch.full((max(int(nbytes), 1),), 255, dtype=torch.uint8, device="cuda")


def test_workspace_contents_do_not_matter():
    """Several slabs per channel: a workspace holding NaN on entry, one
    reused across repeated calls, and one reused for a smaller shape give the
    result of a fresh workspace bit for bit."""
    big = synth.WORKLOADS["bf16_b16_c64_112_w14"]
    d = synth.draw_workload(big, seed=5)
    x, dy = (to_device(d[k], "bf16") for k in ("x", "dy"))
    need = W.wbmm_backward_table_workspace_bytes(x.shape, 14, x.dtype)
    assert need > 0
    ref = W.wbmm_backward_table(x, dy, 14, workspace=W.new_workspace(need))
    ws = garbage_workspace(need)
    for _ in range(3):
        got = W.wbmm_backward_table(x, dy, 14, workspace=ws)
        _, got2 = W.wbmm_backward(x, dy, to_device(d["t"], "bf16"), 14, workspace=ws)
        torch.cuda.synchronize()
        assert torch.equal(got, ref) and torch.equal(got2, ref)
    xs, dys = x[:, :48].contiguous(), dy[:, :48].contiguous()
    small = W.wbmm_backward_table(xs, dys, 14, workspace=ws)
    fresh = W.wbmm_backward_table(xs, dys, 14, workspace=garbage_workspace(need))
    torch.cuda.synchronize()
    assert torch.equal(small, fresh)
    # the slab split depends on the channel count: the same products, summed
    # in another order
    assert float((small - ref[:48]).abs().max()) <= 1e-5 * float(ref[:48].abs().max())


# ------------------------------------------------------------- hierarchical

HIER = [
    # (B, C, H, W, wl): global windows 2 wl, ragged and padded maps; maps
    # tiled by 2 wl >= 10 take the one-pass table gradients (one or several
    # slabs per channel), the others two table-gradient launches
    (2, 3, 28, 28, 7),
    (16, 3, 28, 28, 7),
    (16, 1, 32, 32, 8),
    (4, 2, 20, 20, 5),
    (4, 2, 14, 14, 7),     # 196-element images: row-kernel forward, channel-stream backward
    (1, 2, 30, 17, 7),
    (2, 2, 16, 16, 4),
    (1, 2, 21, 35, 5),
    (2, 1, 32, 32, 8),
    (2, 2, 12, 20, 3),
    (3, 2, 8, 12, 2),
    (2, 2, 6, 6, 1),
    (1, 2, 12, 12, 6),
]


def draw_hier(B, C, H, Wd, wl, dtype, seed):
    d = draw(B, C, H, Wd, 2 * wl, dtype, seed=seed)
    r = np.random.default_rng(seed + 1000)
    d["tl"], d["tl64"] = synth.round_to(0.02 * r.standard_normal((C, (2 * wl - 1) ** 2)), dtype)
    return d


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("shape", HIER, ids=lambda s: "B%dC%dH%dW%dwl%d" % s)
def test_hier_parity(shape, dtype):
    B, C, H, Wd, wl = shape
    d = draw_hier(B, C, H, Wd, wl, dtype, seed=31)
    x, tg, tl, dy = (to_device(d[k], dtype) for k in ("x", "t", "tl", "dy"))
    y = W.wbmm_hier_forward(x, tg, tl, wl)
    dx, dtg, dtl = W.wbmm_hier_backward(x, dy, tg, tl, wl)
    dx2 = W.wbmm_hier_backward_input(dy, tg, tl, wl)
    torch.cuda.synchronize()
    assert torch.equal(dx, dx2)
    want = {"fwd": oracle.hier_forward(d["x64"], d["t64"], d["tl64"], wl),
            "dx": oracle.hier_backward_input(d["dy64"], d["t64"], d["tl64"], wl)}
    want["dtg"], want["dtl"] = oracle.hier_backward_tables(d["x64"], d["dy64"], wl)
    got = {"fwd": to_f64(y), "dx": to_f64(dx), "dtg": to_f64(dtg), "dtl": to_f64(dtl)}
    check(got, want, dtype, "hier %s %s" % (dtype, shape))


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("wl", [2, 3, 7])
def test_hier_integer_data_bit_exact(wl, dtype):
    """Small integers in both tables and the data: every sum is exact in fp32
    and below 256 in magnitude, so the GPU must equal the oracle exactly
    (wl = 7: a tiled map with several slabs per channel, the one-pass table
    gradients)."""
    B, C, H, Wd = (3, 2, 5 * wl, 4 * wl + 1) if wl < 7 else (16, 2, 28, 28)
    r = np.random.default_rng(40 + wl)
    d = {}
    for k, shp in (("x", (B, C, H, Wd)), ("dy", (B, C, H, Wd)), ("t", (C, (4 * wl - 1) ** 2)),
                   ("tl", (C, (2 * wl - 1) ** 2))):
        d[k], d[k + "64"] = synth.round_to(r.integers(-1, 2, size=shp).astype(np.float64), dtype)
    x, tg, tl, dy = (to_device(d[k], dtype) for k in ("x", "t", "tl", "dy"))
    y = W.wbmm_hier_forward(x, tg, tl, wl)
    dx, dtg, dtl = W.wbmm_hier_backward(x, dy, tg, tl, wl)
    torch.cuda.synchronize()
    assert np.array_equal(to_f64(y), oracle.hier_forward(d["x64"], d["t64"], d["tl64"], wl))
    assert np.array_equal(to_f64(dx), oracle.hier_backward_input(d["dy64"], d["t64"], d["tl64"], wl))
    wg_, wl_ = oracle.hier_backward_tables(d["x64"], d["dy64"], wl)
    assert np.array_equal(to_f64(dtg), wg_) and np.array_equal(to_f64(dtl), wl_)


@pytest.mark.parametrize("name", list(synth.HIER_WORKLOADS))
def test_hier_workload_full_size(name):
    """The hierarchical workloads at full size, as the benchmark launches them,
    against the oracle on every channel.  The one-pass table gradients also
    agree with the two single-scale table gradients (other summation order:
    to 1e-5 of the largest entry)."""
    wl = synth.HIER_WORKLOADS[name]
    wloc = wl.w // 2
    d = synth.draw_workload(wl, seed=0)
    d["tl"], d["tl64"] = synth.draw_local_table(wl.C, wloc, wl.dtype, seed=0)
    print("[workload] %s" % name, flush=True)
    x, tg, tl, dy = (to_device(d[k], wl.dtype) for k in ("x", "t", "tl", "dy"))
    y = W.wbmm_hier_forward(x, tg, tl, wloc)
    dx, dtg, dtl = W.wbmm_hier_backward(x, dy, tg, tl, wloc)
    sg = W.wbmm_backward_table(x, dy, 2 * wloc)
    sl = W.wbmm_backward_table(x, dy, wloc)
    torch.cuda.synchronize()
    for a, b in ((dtg, sg), (dtl, sl)):
        assert float((a - b).abs().max()) <= 1e-5 * float(b.abs().max())
    want = {"fwd": oracle.hier_forward(d["x64"], d["t64"], d["tl64"], wloc),
            "dx": oracle.hier_backward_input(d["dy64"], d["t64"], d["tl64"], wloc)}
    want["dtg"], want["dtl"] = oracle.hier_backward_tables(d["x64"], d["dy64"], wloc)
    got = {"fwd": to_f64(y), "dx": to_f64(dx), "dtg": to_f64(dtg), "dtl": to_f64(dtl)}
    for k, v in got.items():
        assert np.isfinite(v).all(), "%s %s: non-finite output" % (name, k)
    check(got, want, wl.dtype, name)


def test_hier_workspace_contents_do_not_matter():
    """The one-pass hierarchical backward with several slabs per channel: a
    workspace holding NaN on entry, reused across repeated calls and for a
    smaller shape in between, equals a fresh workspace bit for bit."""
    wl = synth.HIER_WORKLOADS["bf16_b16_c64_112_hier7"]
    d = synth.draw_workload(wl, seed=6)
    d["tl"], d["tl64"] = synth.draw_local_table(wl.C, 7, wl.dtype, seed=6)
    x, tg, tl, dy = (to_device(d[k], wl.dtype) for k in ("x", "t", "tl", "dy"))
    need = W.wbmm_hier_backward_workspace_bytes(x.shape, 7, x.dtype)
    ref = W.wbmm_hier_backward(x, dy, tg, tl, 7, workspace=W.new_workspace(need))
    ws = garbage_workspace(need)
    for _ in range(3):
        got = W.wbmm_hier_backward(x, dy, tg, tl, 7, workspace=ws)
        W.wbmm_hier_backward(x[:4, :16].contiguous(), dy[:4, :16].contiguous(), tg[:16].contiguous(),
                             tl[:16].contiguous(), 7, workspace=ws)
        torch.cuda.synchronize()
        for a, b in zip(got, ref):
            assert torch.equal(a, b)


def test_hier_autograd_and_zero_tables():
    d = draw_hier(2, 3, 14, 21, 7, "f32", seed=33)
    x = to_device(d["x"], "f32").requires_grad_(True)
    tg = to_device(d["t"], "f32").requires_grad_(True)
    tl = to_device(d["tl"], "f32").requires_grad_(True)
    dy = to_device(d["dy"], "f32")
    y = W.wbmm_hier(x, tg, tl, 7)
    y.backward(dy)
    torch.cuda.synchronize()
    want = {"fwd": oracle.hier_forward(d["x64"], d["t64"], d["tl64"], 7),
            "dx": oracle.hier_backward_input(d["dy64"], d["t64"], d["tl64"], 7)}
    want["dtg"], want["dtl"] = oracle.hier_backward_tables(d["x64"], d["dy64"], 7)
    check({"fwd": to_f64(y), "dx": to_f64(x.grad), "dtg": to_f64(tg.grad), "dtl": to_f64(tl.grad)},
          want, "f32", "hier autograd")
    # zero tables: the two identity shortcuts alone, y = 2 x exactly
    xb = to_device(d["x"], "f32")
    z = W.wbmm_hier_forward(xb, torch.zeros_like(tg), torch.zeros_like(tl), 7)
    torch.cuda.synchronize()
    assert torch.equal(z, 2 * xb)


# ------------------------------------------------ cached-matrix (dense) form

DENSE = [
    # (B, C, H, W, wh, ww): rectangular and square windows, ragged maps
    (2, 3, 9, 10, 3, 5),
    (1, 2, 14, 21, 7, 7),
    (2, 2, 28, 28, 14, 14),
    (1, 2, 20, 17, 16, 8),
    (3, 2, 5, 9, 2, 3),
    (2, 1, 16, 32, 16, 16),
    (1, 3, 7, 7, 1, 7),
]


def dense_draw(B, C, H, Wd, wh, ww, dtype, seed):
    r = np.random.default_rng(seed)
    d = {}
    for k, shp, sd in (("x", (B, C, H, Wd), 1.0), ("dy", (B, C, H, Wd), 1.0),
                       ("t", (C, (2 * wh - 1) * (2 * ww - 1)), 0.02),
                       ("m", (C, wh * ww, wh * ww), 0.05)):
        d[k], d[k + "64"] = synth.round_to(sd * r.standard_normal(shp), dtype)
    return d


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("shape", DENSE, ids=lambda s: "B%dC%dH%dW%dw%dx%d" % s)
def test_dense_form_parity(shape, dtype):
    """An arbitrary (non-Toeplitz) per-channel matrix: forward, input gradient
    and matrix gradient against the oracle; the matrix built from a table is
    the table gathered bit for bit, and the rectangular-window WBMM composed
    from it matches the oracle's table form in all three passes."""
    B, C, H, Wd, wh, ww = shape
    d = dense_draw(B, C, H, Wd, wh, ww, dtype, seed=51)
    x, dy, t, m = (to_device(d[k], dtype) for k in ("x", "dy", "t", "m"))
    got = {"fwd": W.wbmm_dense_forward(x, m, wh, ww), "dx": W.wbmm_dense_backward_input(dy, m, wh, ww),
           "dm": W.wbmm_dense_backward_matrix(x, dy, wh, ww)}
    mb = W.wbmm_build_matrix(t, wh, ww)
    rect = {"fwd": W.wbmm_rect_forward(x, t, wh, ww), "dx": W.wbmm_rect_backward_input(dy, t, wh, ww),
            "dt": W.wbmm_rect_backward_table(x, dy, wh, ww)}
    torch.cuda.synchronize()
    want = {"fwd": oracle.dense_forward(d["x64"], d["m64"], (wh, ww)),
            "dx": oracle.dense_backward_input(d["dy64"], d["m64"], (wh, ww)),
            "dm": oracle.dense_backward_matrix(d["x64"], d["dy64"], (wh, ww))}
    check({k: to_f64(v) for k, v in got.items()}, want, dtype, "dense %s %s" % (dtype, shape))
    assert np.array_equal(to_f64(mb), oracle.build_matrix(d["t64"], (wh, ww)))
    want_r = {"fwd": oracle.forward(d["x64"], d["t64"], (wh, ww)),
              "dx": oracle.backward_input(d["dy64"], d["t64"], (wh, ww)),
              "dt": oracle.backward_table(d["x64"], d["dy64"], (wh, ww))}
    check({k: to_f64(v) for k, v in rect.items()}, want_r, dtype, "rect %s %s" % (dtype, shape))


def test_dense_bin_matrix_exact():
    """Folding an integer-valued matrix onto the table: exact sums."""
    r = np.random.default_rng(52)
    for wh, ww in ((3, 5), (7, 7), (16, 2)):
        dm64 = r.integers(-4, 5, size=(3, wh * ww, wh * ww)).astype(np.float64)
        got = W.wbmm_bin_matrix(torch.from_numpy(dm64.astype(np.float32)).cuda(), wh, ww)
        torch.cuda.synchronize()
        assert np.array_equal(to_f64(got), oracle.bin_matrix(dm64, (wh, ww)))


# -------------------------------------------------------------- seeded sweep

def sweep_shapes(n, seed, ncu=256):
    """Seeded random shapes: windows 2..16 on ragged maps and on maps the
    windows tile (bands of one image or whole images per 16-window
    sub-tile), channel counts on either side of the compute-unit count (the
    launch plans that split channels into slabs, stream them, take rounds or
    runs of stages, or fall back to the four-wave kernels)."""
    r = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        w = int(r.integers(2, 17))
        if r.random() < 0.6:
            H, Wd = int(r.integers(1, 5)) * w, int(r.choice([1, 2, 4])) * w
        else:
            H, Wd = int(r.integers(1, 3 * w + 1)), int(r.integers(1, 3 * w + 1))
        C = int(r.choice([1, 2, 5, 33, ncu - 3, ncu + 5, ncu + ncu // 2 + 7]))
        B = int(r.integers(1, 9 if C < 64 else 3))
        out.append((B, C, H, Wd, w))
    return out


SWEEP = sweep_shapes(24, 2026)


@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("shape", SWEEP, ids=lambda s: "B%dC%dH%dW%dw%d" % s)
def test_seeded_shape_sweep(shape, dtype):
    """Every pass against the oracle, and the fused backward equal to the
    separate entry points bit for bit, on the seeded random shapes."""
    B, C, H, Wd, w = shape
    d = draw(B, C, H, Wd, w, dtype, seed=B * 7919 + C * 31 + H * 7 + Wd + w)
    label = "sweep %s %s" % (dtype, shape)
    check(run_gpu(d, w, dtype), run_oracle(d, w), dtype, label)
    check_fused(d, w, dtype, label)
