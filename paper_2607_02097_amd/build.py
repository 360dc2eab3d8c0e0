"""Build the WBMM HIP library (libwbmm.so) in-tree for gfx950 with hipcc.

Usage: python -m paper_2607_02097_amd.build   (or call build()).
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import time
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libwbmm.so")
OBJ_DIR = os.path.join(PKG, "_build")

ARCH = "gfx950"
# Packed fp32 VALU forms are kept out of generated code on purpose.
HIP_FLAGS = ["--offload-arch=" + ARCH, "-O3", "-std=c++20", "-fPIC",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-I" + INCLUDE, "-I" + CSRC]

# (source, extra defines): the kernel templates are instantiated once per
# (dtype, window range) so the translation units compile in parallel.
UNITS = [("wbmm_inst.hip", ["-DWBMM_INST_TAG=%s" % tag, "-DWBMM_INST_LO=%d" % lo])
         for tag in ("TagBF16", "TagF32", "TagF16") for lo in (9, 1)]
UNITS += [("wbmm_dense.hip", []), ("wbmm_dispatch.cpp", []), ("wbmm_api.cpp", [])]


def hipcc() -> str:
    p = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(p):
        raise RuntimeError("hipcc not found; the WBMM library needs ROCm's hipcc")
    return p


def _compile(unit) -> str:
    src, defs = unit
    tag = "_".join(d.split("=")[1] for d in defs)
    obj = os.path.join(OBJ_DIR, os.path.basename(src) + (("." + tag) if tag else "") + ".o")
    cmd = [hipcc()] + HIP_FLAGS + defs + ["-c", os.path.join(CSRC, src), "-o", obj]
    if src.endswith(".cpp"):
        cmd = [hipcc(), "-O2", "-std=c++20", "-fPIC", "-I" + INCLUDE, "-I" + CSRC,
               "-D__HIP_PLATFORM_AMD__", "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed for %s:\n%s\n%s" % (src, " ".join(cmd), r.stderr))
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(OBJ_DIR, exist_ok=True)
    t0 = time.time()
    jobs = max(1, min(len(UNITS), int(os.environ.get("MAX_JOBS", os.cpu_count() or 4))))
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(_compile, UNITS))
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [hipcc(), "--offload-arch=" + ARCH, "-shared", "-fPIC"] + objs + ["-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n%s\n%s" % (" ".join(cmd), r.stderr))
    os.replace(tmp, LIB)
    if verbose:
        print("built %s in %.1fs" % (LIB, time.time() - t0))
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
