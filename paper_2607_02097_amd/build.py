"""Build the WBMM HIP library (libwbmm.so) in-tree for gfx950 with hipcc.

Usage: python -m paper_2607_02097_amd.build   (or call build()).

After compiling, the device code of every HIP object is disassembled and the
build fails if any instruction reaches memory through the flat address space:
the kernels address on-chip LDS with ds_* instructions and device memory with
global_* instructions only (a flat access to LDS beyond 64 KB faults).
"""
from __future__ import annotations

import os
import re
import shutil
import subprocess
import sys
import tempfile
import time
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libwbmm.so")
OBJ_DIR = os.path.join(PKG, "_build")
LLVM_BIN = "/opt/rocm/llvm/bin"

ARCH = "gfx950"
# Packed fp32 VALU forms are kept out of generated code on purpose.
HIP_FLAGS = ["--offload-arch=" + ARCH, "-O3", "-std=c++20", "-fPIC",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-I" + INCLUDE, "-I" + CSRC]

# (source, extra defines): the kernel templates are instantiated once per
# (dtype, range of four window sizes) so the translation units compile in
# parallel; the largest windows (slowest units) first.
UNITS = [("wbmm_inst.hip", ["-DWBMM_INST_TAG=%s" % tag, "-DWBMM_INST_LO=%d" % lo])
         for lo in (13, 9, 5, 1) for tag in ("TagBF16", "TagF16", "TagF32")]
UNITS += [("wbmm_dense.hip", []), ("wbmm_reduce.hip", []), ("wbmm_noalloc.hip", []), ("wbmm_dispatch.cpp", []), ("wbmm_api.cpp", [])]


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


def device_disassembly(obj: str) -> str:
    """The gfx950 device code of one HIP object file, disassembled."""
    tool = lambda n: os.path.join(LLVM_BIN, n)
    with tempfile.TemporaryDirectory() as td:
        fb, co = os.path.join(td, "fatbin"), os.path.join(td, "dev.co")
        subprocess.run([tool("llvm-objcopy"), "--dump-section=.hip_fatbin=" + fb, obj],
                       check=True, capture_output=True)
        subprocess.run([tool("clang-offload-bundler"), "--unbundle", "--type=o", "--input=" + fb,
                        "--targets=hipv4-amdgcn-amd-amdhsa--" + ARCH, "--output=" + co],
                       check=True, capture_output=True)
        r = subprocess.run([tool("llvm-objdump"), "-d", "--mcpu=" + ARCH, co],
                           check=True, capture_output=True, text=True)
        return r.stdout


def flat_accesses(disasm: str) -> list:
    """(kernel symbol, instruction) of every flat-address-space access."""
    out, sym = [], "?"
    for line in disasm.splitlines():
        m = re.match(r"^[0-9a-f]+ <(.+)>:$", line)
        if m:
            sym = m.group(1)
            continue
        m = re.search(r"\b(flat_[a-z0-9_]+)\b", line)
        if m:
            out.append((sym, m.group(1)))
    return out


def check_no_flat(objs) -> None:
    bad = []
    for o in objs:
        if o.endswith(".hip.o") or ".hip." in os.path.basename(o):
            bad += [(os.path.basename(o),) + f for f in flat_accesses(device_disassembly(o))]
    if bad:
        lines = "\n".join("  %s: %s in %s" % (o, ins, sym) for o, sym, ins in bad[:20])
        raise RuntimeError("device code reaches memory through flat instructions "
                           "(%d found); every LDS pointer must stay in the local "
                           "address space:\n%s" % (len(bad), lines))


def build(verbose: bool = False) -> str:
    os.makedirs(OBJ_DIR, exist_ok=True)
    t0 = time.time()
    jobs = max(1, min(len(UNITS), int(os.environ.get("MAX_JOBS", os.cpu_count() or 4))))
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(_compile, UNITS))
    check_no_flat(objs)
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
