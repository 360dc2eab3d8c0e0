"""Seeded synthetic inputs for WBMM workloads.

This module only draws random numbers and rounds them to a storage dtype; it
contains none of the operator's arithmetic.  Both the HIP path and the CPU
oracle receive exactly the values produced here.

Recipe (one fixed order, so every consumer sees the same values):
  rng = numpy.random.default_rng(seed)            # PCG64
  x   = rng.standard_normal((B, C, H, W))          # activations ~ N(0, 1)
  t   = 0.02 * rng.standard_normal((C, (2w-1)^2))  # table ~ N(0, 0.02^2)
  dy  = rng.standard_normal((B, C, H, W))          # upstream gradient ~ N(0, 1)
then each array is rounded once to the storage dtype with round-to-nearest-even
(fp64 -> fp32 for "f32"; fp64 -> fp32 -> bf16 for "bf16"; fp64 -> fp16 for
"f16").  ``*_64`` holds the rounded values widened back to float64.

The workloads stand in for the stage shapes of the paper's models (operator
benchmark at 256 channels; WBMM-S stage widths 96/192/384; Pico width 64) with
activations drawn from N(0, 1); no dataset is read.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    dtype: str          # "f32" | "bf16" | "f16"
    B: int
    C: int
    H: int
    W: int
    w: int
    passes: tuple       # subset of ("fwd", "dx", "dt"); hierarchical: ("hfwd", "hbwd")
    hier: bool = False  # hierarchical form: global windows w, local w / 2

    @property
    def table_len(self) -> int:
        return (2 * self.w - 1) ** 2

    @property
    def windows_per_channel(self) -> int:
        nh = -(-self.H // self.w)
        nw = -(-self.W // self.w)
        return self.B * nh * nw

    def flops(self, passes=None) -> float:
        """Algorithmic flops, 2*C*N*d^2 per pass (no padding, no re-reads).
        Hierarchical form: the forward and the input gradient are products
        with the d x d fused matrix; the table gradients are those of the two
        scales (the local one a quarter of the global one)."""
        d = self.w * self.w
        per = 2.0 * self.C * self.windows_per_channel * d * d
        total = 0.0
        for p in (passes if passes is not None else self.passes):
            total += per * {"hbwd": 2.25}.get(p, 1.0)
        return total


# The five workloads: parity small case, w=7 memory-bound forward, and three
# w=14 forward+backward stage shapes.
WORKLOADS = {
    "f32_b1_c8_28_w7": Workload("f32_b1_c8_28_w7", "f32", 1, 8, 28, 28, 7, ("fwd", "dx", "dt")),
    "bf16_b64_c96_56_w7": Workload("bf16_b64_c96_56_w7", "bf16", 64, 96, 56, 56, 7, ("fwd",)),
    "bf16_b64_c192_28_w14": Workload("bf16_b64_c192_28_w14", "bf16", 64, 192, 28, 28, 14, ("fwd", "dx", "dt")),
    "bf16_b128_c384_14_w14": Workload("bf16_b128_c384_14_w14", "bf16", 128, 384, 14, 14, 14, ("fwd", "dx", "dt")),
    "bf16_b16_c64_112_w14": Workload("bf16_b16_c64_112_w14", "bf16", 16, 64, 112, 112, 14, ("fwd", "dx", "dt")),
}


# Hierarchical form (global 14 x 14 windows, local 7 x 7 sub-windows): the
# headline stage shape, and a Pico-width map at dense-prediction resolution.
HIER_WORKLOADS = {
    "bf16_b64_c192_28_hier7": Workload("bf16_b64_c192_28_hier7", "bf16", 64, 192, 28, 28, 14,
                                       ("hfwd", "hbwd"), hier=True),
    "bf16_b16_c64_112_hier7": Workload("bf16_b16_c64_112_hier7", "bf16", 16, 64, 112, 112, 14,
                                       ("hfwd", "hbwd"), hier=True),
}


def draw_local_table(C: int, wl: int, dtype: str, seed: int = 0):
    """Seeded local table of the hierarchical form, N(0, 0.02^2), as
    (stored, float64) like draw()."""
    r = np.random.default_rng(seed + 7919)
    return round_to(0.02 * r.standard_normal((C, (2 * wl - 1) ** 2)), dtype)


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even); returns the
    16-bit patterns as uint16.  NaN stays NaN (quiet bit set)."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        r[nan] = ((u[nan] >> 16) | 0x40).astype(np.uint16)
    return r


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    u = np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return u.view(np.float32).astype(np.float64)


def round_to(a64: np.ndarray, dtype: str):
    """Round fp64 values to ``dtype``; returns (storage array, fp64 view of the
    rounded values).  Storage: float32, uint16 bit patterns (bf16), float16."""
    if dtype == "f32":
        s = a64.astype(np.float32)
        return s, s.astype(np.float64)
    if dtype == "bf16":
        s = f32_to_bf16_bits(a64.astype(np.float32))
        return s, bf16_bits_to_f64(s)
    if dtype == "f16":
        s = a64.astype(np.float16)
        return s, s.astype(np.float64)
    raise ValueError("unknown dtype %r" % dtype)


def draw(B, C, H, W, w, dtype="f32", seed=0, t_std=0.02):
    """Draw (x, t, dy) in the fixed order above and round them to ``dtype``.

    Returns a dict with storage arrays ``x, t, dy`` and fp64 copies of the
    rounded values ``x64, t64, dy64``.  ``w`` may be an int or (wh, ww)."""
    wh, ww = (w, w) if isinstance(w, int) else (int(w[0]), int(w[1]))
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((B, C, H, W))
    t = t_std * rng.standard_normal((C, (2 * wh - 1) * (2 * ww - 1)))
    dy = rng.standard_normal((B, C, H, W))
    out = {}
    for name, a in (("x", x), ("t", t), ("dy", dy)):
        s, r = round_to(a, dtype)
        out[name] = s
        out[name + "64"] = r
    return out


def draw_workload(wl: Workload, seed=0):
    return draw(wl.B, wl.C, wl.H, wl.W, wl.w, wl.dtype, seed)
