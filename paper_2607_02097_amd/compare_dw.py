"""Operator comparison on one MI355X: WBMM forward vs depthwise convolution.

Context for the operator-level benchmark of the paper (single layer, 256
channels, batch sizes 4..256, feature maps 14..112): standard depthwise
convolution (PyTorch-ROCm ``conv2d`` with groups = C and "same" zero padding,
i.e. MIOpen) with kernels 5, 13 and 27, against the WBMM forward kernel of
this package with 7 x 7 and 14 x 14 windows, on the same input tensor.  This
is a comparison harness, not part of the operator: the convolution is the
comparison system the paper measures against.

Throughput is reported in thousands of images per second (kFPS = B / time),
each configuration timed with HIP events after a warm-up: the WBMM kernel
around replays of a captured graph of 20 launches (the kernels are short; a
graph removes the Python launch cost), the convolution around eager launches
(MIOpen's kernels are long).  One JSON line per (map, method).

Usage: python -m paper_2607_02097_amd.compare_dw [--dtype f32] [--batch 128]
                                                 [--maps 14,28,56,112]
"""
from __future__ import annotations

import argparse
import json
import sys

import torch

from . import binding as W

DW_KERNELS = (5, 13, 27)
WBMM_WINDOWS = (7, 14)


def _time(fn, graph: bool, reps=20, rounds=10):
    """Average time of fn (ms): HIP events around `rounds` replays of a graph
    of `reps` launches (graph=True) or around rounds x reps eager launches;
    slow calls (> 5 ms) are timed over 5 eager launches."""
    fn()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    fn()
    b.record()
    torch.cuda.synchronize()
    if a.elapsed_time(b) > 5.0:
        reps, rounds, graph = 1, 5, False
    g = None
    if graph:
        g = torch.cuda.CUDAGraph()
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.graph(g, stream=s):
            for _ in range(reps):
                fn()
        torch.cuda.current_stream().wait_stream(s)
        g.replay()
        torch.cuda.synchronize()
    a.record()
    for _ in range(rounds):
        if g is not None:
            g.replay()
        else:
            for _ in range(reps):
                fn()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / (rounds * reps), ("graph" if g is not None else "eager")


def run(dtype: str, batch: int, maps, channels: int = 256):
    tdt = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[dtype]
    dev = torch.device("cuda:0")
    gen = torch.Generator(device=dev).manual_seed(0)
    rows = []
    for hw in maps:
        x = torch.randn((batch, channels, hw, hw), device=dev, generator=gen).to(tdt)
        base = None
        for k in DW_KERNELS:
            wgt = (0.02 * torch.randn((channels, 1, k, k), device=dev, generator=gen)).to(tdt)
            ms, mode = _time(lambda: torch.nn.functional.conv2d(x, wgt, padding=k // 2, groups=channels), False)
            if k == 5:
                base = ms
            rows.append({"map": hw, "method": "DW-Std %dx%d" % (k, k), "ms": round(ms, 4),
                         "kfps": round(batch / ms, 2), "speedup_vs_dw5": round(base / ms, 3), "launch": mode})
        for w in WBMM_WINDOWS:
            t = (0.02 * torch.randn((channels, (2 * w - 1) ** 2), device=dev, generator=gen)).to(tdt)
            y = torch.empty_like(x)
            ms, mode = _time(lambda: W.wbmm_forward(x, t, w, out=y), True)
            rows.append({"map": hw, "method": "WBMM %dx%d" % (w, w), "ms": round(ms, 4),
                         "kfps": round(batch / ms, 2), "speedup_vs_dw5": round(base / ms, 3), "launch": mode})
        del x
        torch.cuda.empty_cache()
    for r in rows:
        r.update({"dtype": dtype, "batch": batch, "channels": channels})
        print(json.dumps(r), flush=True)
    return rows


def main(argv=None):
    p = argparse.ArgumentParser()
    p.add_argument("--dtype", default="f32", choices=["f32", "bf16", "f16"])
    p.add_argument("--batch", type=int, default=128)
    p.add_argument("--maps", default="14,28,56,112")
    a = p.parse_args(argv)
    W.load_library()
    run(a.dtype, a.batch, [int(m) for m in a.maps.split(",")])


if __name__ == "__main__":
    sys.exit(main())
