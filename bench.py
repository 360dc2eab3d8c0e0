#!/usr/bin/env python3
"""Benchmark of the WBMM hot path on one MI355X.

One step = forward + input gradient + table gradient (all three passes of the
operator) over one batch of seeded synthetic input already resident in device
memory: the forward kernel, then the fused backward kernel, which computes
both gradients from one read of x and dy.  The headline workload is the w=14
stage shape B=64, C=192, H=W=28 in bfloat16 with float32 accumulation.  The
separate input- and table-gradient kernels are timed as well and reported
beside the step (per_pass_ms).

Prints ONE JSON line with the throughput (algorithmic TFLOP/s, 6*C*N*d^2 per
step), the roofline of the dominant kernel (timed live with HIP events on the
stream the kernels run on) and the fp64 CPU oracle timed on the host cores.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0      # MI355X HBM3E
BF16_PEAK_TFLOPS = 2516.6  # MI355X dense bf16/fp16 matrix-core peak
F32_PEAK_TFLOPS = 157.3    # MI355X fp32 matrix/vector peak
HEADLINE = "bf16_b64_c192_28_w14"
METRIC = "WBMM fwd+bwd TFLOP/s & % bf16 MFMA peak, B=64 C=192 28² w=14"


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=2000)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--workload", default=HEADLINE)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cold", action="store_true",
                   help="rotate through enough input sets to defeat the 256 MB Infinity Cache")
    p.add_argument("--one-mode", action="store_true",
                   help="measure only the headline cache mode (hardware-counter runs)")
    p.add_argument("--eager", action="store_true",
                   help="launch without HIP graphs (for hardware-counter runs)")
    p.add_argument("--calibrate-copy", type=int, default=0, metavar="BYTES",
                   help="only run a plain device copy of BYTES bytes (counter calibration)")
    return p.parse_args()


# HBM traffic of the dominant kernel, from two rocprofv3 --pmc runs (FETCH_SIZE,
# WRITE_SIZE; KiB per dispatch) scaled by what the same counters read for a
# plain copy of known size.  Valid only for the kernel source it was measured
# on (sha256 of the kernel header's code without comments and blank lines);
# otherwise reported as null.
TRAFFIC = {
    ("bf16_b128_c384_14_w14", "bwd"): {"source": "c5c88ade4f762eae", "bytes": 60216951},
    ("bf16_b128_c384_14_w14", "dt"): {"source": "c5c88ade4f762eae", "bytes": 40341241},
    ("bf16_b128_c384_14_w14", "dx"): {"source": "c5c88ade4f762eae", "bytes": 39186822},
    ("bf16_b128_c384_14_w14", "fwd"): {"source": "c5c88ade4f762eae", "bytes": 39195548},
    ("bf16_b16_c64_112_hier7", "hbwd"): {"source": "c5c88ade4f762eae", "bytes": 79881986},
    ("bf16_b16_c64_112_hier7", "hfwd"): {"source": "c5c88ade4f762eae", "bytes": 51712583},
    ("bf16_b16_c64_112_w14", "bwd"): {"source": "c5c88ade4f762eae", "bytes": 78627980},
    ("bf16_b16_c64_112_w14", "dt"): {"source": "c5c88ade4f762eae", "bytes": 52797942},
    ("bf16_b16_c64_112_w14", "dx"): {"source": "c5c88ade4f762eae", "bytes": 51593424},
    ("bf16_b16_c64_112_w14", "fwd"): {"source": "c5c88ade4f762eae", "bytes": 51586736},
    ("bf16_b64_c192_28_hier7", "hbwd"): {"source": "c5c88ade4f762eae", "bytes": 60621653},
    ("bf16_b64_c192_28_hier7", "hfwd"): {"source": "c5c88ade4f762eae", "bytes": 40013008},
    ("bf16_b64_c192_28_w14", "bwd"): {"source": "c5c88ade4f762eae", "bytes": 59373612},
    ("bf16_b64_c192_28_w14", "dt"): {"source": "c5c88ade4f762eae", "bytes": 39781561},
    ("bf16_b64_c192_28_w14", "dx"): {"source": "c5c88ade4f762eae", "bytes": 39369981},
    ("bf16_b64_c192_28_w14", "fwd"): {"source": "c5c88ade4f762eae", "bytes": 39392765},
    ("bf16_b64_c96_56_w7", "fwd"): {"source": "c5c88ade4f762eae", "bytes": 77247279},
}


def image_layout(wl):
    """Whether the library runs this workload's 16-bit forward (and input
    gradient) with the image-layout kernel (freshly allocated tensors are
    16-byte aligned): windows tile the map, NW is a power of two up to 16, a
    16-window sub-tile is whole bands of one image or whole images."""
    if wl.dtype not in ("bf16", "f16") or wl.H % wl.w or wl.W % wl.w:
        return False
    nh, nw = wl.H // wl.w, wl.W // wl.w
    if nw > 16 or nw & (nw - 1):
        return False
    wpi = nh * nw
    if wpi % 16 == 0:
        return (wl.w * wl.W) % 8 == 0
    if 16 % wpi == 0:
        return (wl.H * wl.W) % 8 == 0 and 2 * (16 // wpi) * wl.C * wl.H * wl.W < 2 ** 31
    return False


def fixed_offset_rows(wl):
    """Whether the gradient kernels address this workload's rows by fixed
    offsets (see the kernel header): windows tile the map, NW a power of two
    up to 16, 16-window sub-tiles are whole bands of one image or whole
    images, and rows start on a dword (float32, or an even window)."""
    if wl.H % wl.w or wl.W % wl.w or (wl.dtype != "f32" and wl.w % 2):
        return False
    nh, nw = wl.H // wl.w, wl.W // wl.w
    if nw > 16 or nw & (nw - 1):
        return False
    es = 4 if wl.dtype == "f32" else 2
    wpi = nh * nw
    if wpi % 16 != 0 and 16 % wpi != 0:
        return False
    if 16 % wpi == 0 and wpi % 16 != 0 and 16 * wl.C * wl.H * wl.W * es >= 2 ** 31:
        return False
    return wl.w * wl.W * 16 * es < 2 ** 31


def kernel_source_hash():
    """Hash of the kernel source without its comments and blank lines, so
    that a comment edit keeps the traffic entries measured on that code."""
    import hashlib
    import re
    path = os.path.join(ROOT, "paper_2607_02097_amd", "csrc", "wbmm_kernels.h")
    code = []
    for line in open(path, encoding="utf-8"):
        line = re.sub(r"//.*", "", line).strip()
        if line:
            code.append(line)
    return hashlib.sha256("\n".join(code).encode()).hexdigest()[:16]


def calibrate_copy(nbytes, steps):
    import torch
    dev = torch.device("cuda:0")
    a = torch.ones(nbytes // 2, dtype=torch.bfloat16, device=dev)
    b = torch.empty_like(a)
    for _ in range(steps):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"calibration": "copy", "bytes_read": a.numel() * 2,
                      "bytes_written": b.numel() * 2, "launches": steps}))


def kernel_names(wl, ncu):
    """Name of each pass's kernel as the profiler prints it (every template
    argument), from the dispatch rules of the library."""
    fk = "wbmm_fwd_img_kernel" if image_layout(wl) else "wbmm_fwd_kernel"
    tl = "true" if fixed_offset_rows(wl) else "false"
    # channel-stream gradients: fixed-offset rows and no more channels than
    # compute units, or (plain form) rounds whose last one is at least half
    # full (a nearly empty last round takes runs of stages where they apply,
    # in no workload here, else the four-wave kernels)
    rem = wl.C % ncu
    chan_stream = fixed_offset_rows(wl) and (wl.C <= ncu or rem == 0 or rem >= ncu // 2)
    hier_stream = fixed_offset_rows(wl) and wl.C <= ncu
    dtk = "wbmm_bwd_stream_kernel" if chan_stream else "wbmm_dt_kernel"
    bwk = "wbmm_bwd_stream_kernel" if chan_stream else "wbmm_bwd_kernel"
    img = fk == "wbmm_fwd_img_kernel"
    fwd_tail = (lambda rev, hier: "<%s,%d," + rev + "," + hier + ">") if img else \
        (lambda rev, hier: "<%s,%d," + rev + "," + hier + "," + (tl if hier == "false" else "false") + ">")
    tag = {"bf16": "TagBF16", "f16": "TagF16", "f32": "TagF32"}[wl.dtype]
    names = {"fwd": fk + fwd_tail("false", "false"), "dx": fk + fwd_tail("true", "false"),
             # stream kernels: <tag, w, dX too, local half-window (0: plain form), copy waves, runs>
             "dt": dtk + ("<%s,%d,false,0,0,false>" if chan_stream else "<%s,%d," + tl + ">"),
             "bwd": bwk + ("<%s,%d,true,0,4,false>" if chan_stream else "<%s,%d," + tl + ">"),
             "hfwd": fk + fwd_tail("false", "true"),
             "hbwd": ("wbmm_bwd_stream_kernel<%s,%d,true," + str(wl.w // 2) + ",0,false>") if hier_stream and wl.w >= 10
                     else "wbmm_hier_backward (several launches) <%s,%d>"}
    return {k: v % (tag, wl.w) for k, v in names.items()}


def pass_bytes(wl, p, es):
    """Algorithmic bytes of one kernel (each tensor touched once)."""
    act = wl.B * wl.C * wl.H * wl.W * es
    tab = wl.C * wl.table_len
    if wl.hier:
        tabs = tab + wl.C * (wl.w - 1) ** 2  # global and local tables
        if p == "hfwd":
            return 2 * act + tabs * es
        return 3 * act + tabs * es + tabs * 4  # read x, dy, tables; write dx, float32 gradients
    if p in ("fwd", "dx"):
        return 2 * act + tab * es          # read input, write output, read table
    if p == "dt":
        return 2 * act + tab * 4           # read x and dy, write float32 dtable
    return 3 * act + tab * es + tab * 4    # fused: read x, dy, table; write dx, dtable


def pass_flops(wl, p):
    return wl.flops(("dx", "dt") if p == "bwd" else (p,))


def run_marks(n, nrun=5):
    """Events that split a timed loop of n iterations into up to nrun runs
    (recorded on the stream inside the timed region: they add no
    synchronisation)."""
    import torch
    nrun = max(1, min(nrun, n))
    bounds = [round(n * (k + 1) / nrun) for k in range(nrun)]
    return [torch.cuda.Event(enable_timing=True) for _ in bounds], bounds


def run_times(start, marks, bounds, per_iter):
    """ms per step of each run between consecutive marks."""
    out, prev, lo = [], start, 0
    for mk, hi in zip(marks, bounds):
        out.append(prev.elapsed_time(mk) / ((hi - lo) * per_iter))
        prev, lo = mk, hi
    return out


def quartiles(v):
    """Median and the first and third quartiles (linear interpolation)."""
    import numpy as np
    q1, q2, q3 = np.percentile(np.asarray(v, dtype=np.float64), [25, 50, 75])
    return float(q2), float(q1), float(q3)


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on one GPU only: the WBMM path shards over channels "
              "with no collective, so there is no multi-GPU step to time "
              "(asked for --gpus %d, WORLD_SIZE=%d)" % (args.gpus, world), file=sys.stderr)
        sys.exit(2)

    if args.calibrate_copy:
        calibrate_copy(args.calibrate_copy, max(args.steps, 1))
        return

    import numpy as np
    import torch

    from paper_2607_02097_amd import binding as W
    from paper_2607_02097_amd import synth

    wl = synth.WORKLOADS.get(args.workload) or synth.HIER_WORKLOADS[args.workload]
    es = 4 if wl.dtype == "f32" else 2
    tdt = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[wl.dtype]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    W.load_library()

    d = synth.draw_workload(wl, seed=0)

    def put(a):
        if wl.dtype == "bf16":
            return torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16).to(dev)
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)

    wloc = wl.w // 2  # local window of the hierarchical form
    if wl.hier:
        d["tl"], d["tl64"] = synth.draw_local_table(wl.C, wloc, wl.dtype, seed=0)

    def make_sets(nsets):
        sets = []
        for _ in range(nsets):
            x, t, dy = put(d["x"]), put(d["t"]), put(d["dy"])
            y, dx = torch.empty_like(x), torch.empty_like(dy)
            dtab = torch.empty((wl.C, wl.table_len), dtype=torch.float32, device=dev)
            if wl.hier:
                tl = put(d["tl"])
                dtl = torch.empty((wl.C, (2 * wloc - 1) ** 2), dtype=torch.float32, device=dev)
                need = W.wbmm_hier_backward_workspace_bytes(x.shape, wloc, tdt)
            else:
                tl = dtl = None
                need = W.wbmm_backward_table_workspace_bytes(x.shape, wl.w, tdt)
            ws = W.new_workspace(need, dev)  # counters start at zero, stay zero
            sets.append((x, t, dy, y, dx, dtab, ws, tl, dtl))
        return sets

    # cold mode: enough input sets (x, dy, y, dx each) that the rotation
    # spans more than twice the 256 MB Infinity Cache
    per_set = 4 * wl.B * wl.C * wl.H * wl.W * es
    n_cold = max(2, int(np.ceil(2 * 256e6 / per_set)) + 1)

    passes = wl.passes
    # kernels of one step: the fused backward covers the two gradients
    step_kernels = ["fwd", "bwd"] if "dt" in passes else list(passes)
    if wl.hier:
        step_kernels = list(passes)
    timed = step_kernels + [p for p in passes if p not in step_kernels and p != "fwd"]
    lib = W.load_library()
    code = W.DTYPE_CODES[tdt]
    import ctypes
    vp = ctypes.c_void_p
    stream = torch.cuda.current_stream(dev)

    def launch(sets, p, i):
        """One pass through the C ABI on torch's current stream (raw pointers,
        no per-call Python checks: the shapes were validated above)."""
        x, t, dy, y, dx, dtab, ws, tl, dtl = sets[i % len(sets)]
        st = vp(torch.cuda.current_stream(dev).cuda_stream)
        dims = (wl.B, wl.C, wl.H, wl.W, wl.w, code, st)
        hdims = (wl.B, wl.C, wl.H, wl.W, wloc, code, st)
        if p == "hfwd":
            r = lib.wbmm_hier_forward(vp(x.data_ptr()), vp(t.data_ptr()), vp(tl.data_ptr()), vp(y.data_ptr()),
                                      *hdims)
        elif p == "hbwd":
            r = lib.wbmm_hier_backward(vp(x.data_ptr()), vp(dy.data_ptr()), vp(t.data_ptr()), vp(tl.data_ptr()),
                                       vp(dx.data_ptr()), vp(dtab.data_ptr()), vp(dtl.data_ptr()),
                                       vp(ws.data_ptr()), ws.numel(), *hdims)
        elif p == "fwd":
            r = lib.wbmm_forward(vp(x.data_ptr()), vp(t.data_ptr()), vp(y.data_ptr()), *dims)
        elif p == "dx":
            r = lib.wbmm_backward_input(vp(dy.data_ptr()), vp(t.data_ptr()), vp(dx.data_ptr()), *dims)
        elif p == "dt":
            r = lib.wbmm_backward_table(vp(x.data_ptr()), vp(dy.data_ptr()), vp(dtab.data_ptr()),
                                        vp(ws.data_ptr()), ws.numel(), *dims)
        else:
            r = lib.wbmm_backward(vp(x.data_ptr()), vp(dy.data_ptr()), vp(t.data_ptr()),
                                  vp(dx.data_ptr()), vp(dtab.data_ptr()), vp(ws.data_ptr()),
                                  ws.numel(), *dims)
        if r != 0:
            raise RuntimeError("%s failed: %s" % (p, W.wbmm_status_string(r)))

    R = 10  # steps per graph (and launches per pass graph)
    reps = max(1, args.steps // R)
    steps = reps * R
    act_bytes = wl.B * wl.C * wl.H * wl.W * es

    def measure(sets):
        """Warm-up, then exactly `steps` timed steps (HIP-graph replay, or
        eager launches), per-pass kernel times and a device copy, all on the
        input sets given (one set: cache-warm; several: rotated, cold)."""
        nsets = len(sets)
        for i in range(args.warmup):
            for p in timed:
                launch(sets, p, i)
        torch.cuda.synchronize()
        # eager timing (includes host launch overhead; reported, not the value)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        n_eager = min(steps, 50)
        e0.record(stream)
        for i in range(n_eager):
            for p in step_kernels:
                launch(sets, p, i)
        e1.record(stream)
        torch.cuda.synchronize()
        eager_ms = e0.elapsed_time(e1) / n_eager

        if args.eager:
            # plain stream launches (hardware-counter runs serialise dispatches)
            def run_step_block(i0):
                for i in range(i0, i0 + R):
                    for p in step_kernels:
                        launch(sets, p, i)

            def run_pass_block(p, i0):
                for i in range(i0, i0 + R):
                    launch(sets, p, i)
        else:
            def capture(seq, per_step, i0):
                g = torch.cuda.CUDAGraph()
                cs = torch.cuda.Stream(dev)
                cs.wait_stream(stream)
                with torch.cuda.graph(g, stream=cs):
                    for i, p in enumerate(seq):
                        launch(sets, p, i0 + i // per_step)
                stream.wait_stream(cs)
                torch.cuda.synchronize()
                return g

            # one graph per distinct rotation phase of the input sets
            nph = nsets if nsets > 1 else 1
            g_step = [capture([p for _ in range(R) for p in step_kernels], len(step_kernels), ph * R)
                      for ph in range(nph)]
            g_pass = {p: [capture([p] * R, 1, ph * R) for ph in range(nph)] for p in timed}

            def run_step_block(i0):
                g_step[(i0 // R) % nph].replay()

            def run_pass_block(p, i0):
                g_pass[p][(i0 // R) % nph].replay()

        # settle: the step replayed for at least 0.2 s (untimed), so the
        # timed region starts at steady clocks
        t_settle = time.perf_counter()
        i = 0
        while time.perf_counter() - t_settle < 0.2:
            run_step_block(i * R)
            i += 1
            if i % 20 == 0:
                torch.cuda.synchronize()
        torch.cuda.synchronize()

        # timed region: exactly `steps` steps bracketed by synchronisation;
        # events on the stream split it into runs
        t_start = torch.cuda.Event(enable_timing=True)
        t_end = torch.cuda.Event(enable_timing=True)
        marks, bounds = run_marks(reps)
        torch.cuda.synchronize()
        t_start.record(stream)
        i = 0
        for mk, bd in zip(marks, bounds):
            while i < bd:
                run_step_block(i * R)
                i += 1
            mk.record(stream)
        t_end.record(stream)
        torch.cuda.synchronize()
        ms_step = t_start.elapsed_time(t_end) / steps
        run_ms = run_times(t_start, marks, bounds, R)
        # each pass alone, timed with HIP events on the stream it runs on:
        # the average duration of one launch of its kernel
        per_pass = {}
        for p in timed:
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            for k in range(reps):
                run_pass_block(p, k * R)
            b.record(stream)
            torch.cuda.synchronize()
            per_pass[p] = a.elapsed_time(b) / (reps * R)
        # a plain device copy of one activation tensor, rotated like the inputs
        scratch = torch.empty_like(sets[0][0])
        ncopy = 10

        def copies():
            for k in range(ncopy):
                scratch.copy_(sets[k % nsets][0])
        if not args.eager:
            g_copy = torch.cuda.CUDAGraph()
            cs = torch.cuda.Stream(dev)
            cs.wait_stream(stream)
            with torch.cuda.graph(g_copy, stream=cs):
                copies()
            stream.wait_stream(cs)
            torch.cuda.synchronize()
            copies = g_copy.replay
        copies()
        torch.cuda.synchronize()
        ca, cb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ncr = max(1, min(reps, 100))
        ca.record(stream)
        for _ in range(ncr):
            copies()
        cb.record(stream)
        torch.cuda.synchronize()
        copy_ms = ca.elapsed_time(cb) / (ncr * ncopy)
        return {"ms_step": ms_step, "run_ms": run_ms, "per_pass": per_pass, "eager_ms": eager_ms,
                "copy_gbps": 2 * act_bytes / (copy_ms * 1e-3) / 1e9, "nsets": nsets}

    # the headline mode first (cache-warm; --cold makes the rotated sets the
    # headline), then the other mode
    warm_sets = make_sets(1)
    cold_sets = warm_sets + make_sets(n_cold - 1) if (args.cold or not args.one_mode) else None
    first = measure(cold_sets if args.cold else warm_sets)
    other = None if args.one_mode else measure(warm_sets if args.cold else cold_sets)
    main_m, warm_m, cold_m = first, (other if args.cold else first), (first if args.cold else other)
    args.steps = steps
    ms_step, run_ms, per_pass = main_m["ms_step"], main_m["run_ms"], main_m["per_pass"]
    nsets = main_m["nsets"]

    flops = wl.flops()
    tflops = flops / (ms_step * 1e-3) / 1e12
    peak = BF16_PEAK_TFLOPS if wl.dtype in ("bf16", "f16") else F32_PEAK_TFLOPS

    # dominant kernel: the step kernel with the largest average duration
    dom = max(step_kernels, key=per_pass.get)
    dom_ms = per_pass[dom]
    dom_bytes = pass_bytes(wl, dom, es)
    dom_flops = pass_flops(wl, dom)
    ai = dom_flops / dom_bytes
    ridge = peak * 1e12 / (HBM_PEAK_GBS * 1e9)
    kernel_name = kernel_names(wl, torch.cuda.get_device_properties(0).multi_processor_count)[dom]
    if ai < ridge:
        achieved = dom_bytes / (dom_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4)}
    else:
        achieved = dom_flops / (dom_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak,
                "unit": "TFLOP/s", "frac": round(achieved / peak, 4)}
    tr = TRAFFIC.get((wl.name, dom))
    traffic = None
    if tr is not None and tr["source"] == kernel_source_hash():
        traffic = tr["bytes"]
    roof.update({"traffic": traffic, "kernel": kernel_name, "pass": dom,
                 "avg_ms": round(dom_ms, 5), "algorithmic_bytes": dom_bytes,
                 "algorithmic_flops": dom_flops})
    copy_gbps = main_m["copy_gbps"]
    roof["copy_gbps"] = round(copy_gbps, 1)
    if roof["bound"] == "hbm":
        roof["frac_of_copy"] = round(roof["achieved"] / copy_gbps, 4)

    # the step against its own roofline: algorithmic flops over algorithmic
    # bytes of the step's kernels, attainable = min(MFMA peak, AI x HBM peak)
    step_bytes = sum(pass_bytes(wl, p, es) for p in step_kernels)
    step_ai = flops / step_bytes
    attain = min(peak, step_ai * HBM_PEAK_GBS / 1e3)
    step_roof = {"flops": flops, "bytes": step_bytes, "ai_flop_per_byte": round(step_ai, 2),
                 "attainable_tflops": round(attain, 1), "frac": round(tflops / attain, 4),
                 "attainable_at_copy_bw_tflops": round(min(peak, step_ai * copy_gbps / 1e3), 1)}
    med, q1, q3 = quartiles(run_ms)
    runs = {"n": len(run_ms), "ms_per_step": [round(v, 5) for v in run_ms],
            "median_ms": round(med, 5), "iqr_ms": [round(q1, 5), round(q3, 5)]}

    def mode_summary(m):
        """Step and dominant-kernel figures of one cache mode."""
        t = flops / (m["ms_step"] * 1e-3) / 1e12
        dms = m["per_pass"][dom]
        ach = dom_bytes / (dms * 1e-3) / 1e9
        mmed, mq1, mq3 = quartiles(m["run_ms"])
        return {"input_sets": m["nsets"], "ms_per_step": round(m["ms_step"], 5), "value": round(t, 3),
                "pct_bf16_mfma_peak": round(100 * t / peak, 3),
                "per_pass_ms": {k: round(v, 5) for k, v in m["per_pass"].items()},
                "runs_median_ms": round(mmed, 5), "runs_iqr_ms": [round(mq1, 5), round(mq3, 5)],
                "dominant": {"kernel": kernel_name, "avg_ms": round(dms, 5), "achieved_gbps": round(ach, 1),
                             "frac_hbm": round(ach / HBM_PEAK_GBS, 4), "copy_gbps": round(m["copy_gbps"], 1),
                             "frac_of_copy": round(ach / m["copy_gbps"], 4)}}

    cpu = None
    if not args.no_cpu_baseline:
        # the oracle over the whole workload, repeated for about 10 s
        import oracle
        reps_cpu, cpu_s = 0, 0.0
        while cpu_s < 10.0 and reps_cpu < 200:
            t0 = time.perf_counter()
            if wl.hier:
                oracle.hier_forward(d["x64"], d["t64"], d["tl64"], wloc)
                oracle.hier_backward_input(d["dy64"], d["t64"], d["tl64"], wloc)
                oracle.hier_backward_tables(d["x64"], d["dy64"], wloc)
            if "fwd" in passes:
                oracle.forward(d["x64"], d["t64"], wl.w)
            if "dx" in passes:
                oracle.backward_input(d["dy64"], d["t64"], wl.w)
            if "dt" in passes:
                oracle.backward_table(d["x64"], d["dy64"], wl.w)
            cpu_s += time.perf_counter() - t0
            reps_cpu += 1
        cpu = {"value": round(reps_cpu * flops / cpu_s / 1e12, 6), "unit": "TFLOP/s",
               "cores": oracle.max_threads(), "kind": "oracle",
               "sample": "whole workload, all passes (%s), fp64, %d runs in %.1f s"
                         % ("+".join(passes), reps_cpu, cpu_s)}

    out = {
        "metric": METRIC if args.workload == HEADLINE else "WBMM %s TFLOP/s, %s" % ("+".join(passes), args.workload),
        "value": round(tflops, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic (seeded N(0,1) activations/gradients, N(0,0.02^2) table)",
        "config": {"workload": wl.name, "B": wl.B, "C": wl.C, "H": wl.H, "W": wl.W, "w": wl.w,
                   "passes": list(passes), "step_kernels": step_kernels,
                   "cold_cache": bool(args.cold), "input_sets": nsets},
        "pct_bf16_mfma_peak": round(100 * tflops / peak, 3),
        "per_pass_ms": {k: round(v, 5) for k, v in per_pass.items()},
        "launch": "eager stream launches" if args.eager else "HIP graph replay, %d steps per graph" % R,
        "eager_ms_per_step": round(main_m["eager_ms"], 5),
        "roofline": roof,
        "step_roofline": step_roof,
        "runs": runs,
        "warm": mode_summary(warm_m) if warm_m else None,
        "cold": mode_summary(cold_m) if cold_m else None,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out))


if __name__ == "__main__":
    main()
