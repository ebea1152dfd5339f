"""Build libattr.so (HIP kernels for gfx950 + the C-ABI layer) in-tree.

Usage: python -m paper_2606_11660_amd.build   (or call build()).
Every call recompiles from source; the shared library lands next to this
file so that it travels with the source tree.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import re
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libattr.so")
ARCH = "gfx950"
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")

HIP_SOURCES = ["project.hip", "rowwise.hip", "syrk.hip", "apply_full.hip", "score.hip", "probe.hip"]
CXX_SOURCES = ["api.cpp"]

COMMON = ["-O3", "-fPIC", "-std=c++17", f"-I{INCLUDE}", f"-I{CSRC}", "-Wall",
          "-Wno-unused-function"]
# Packed fp32 ops are disabled for all device code.
DEVICE = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


def _run(cmd):
    p = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in p.stdout.splitlines()
                    if "packed-fp32-ops' is not a recognized feature" not in l)
    if p.returncode != 0:
        raise RuntimeError(f"command failed ({p.returncode}): {' '.join(cmd)}\n{out}")
    return out


def _sgprs(tok: str) -> set:
    m = re.match(r"s\[(\d+):(\d+)\]", tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.match(r"s(\d+)$", tok)
    return {int(m.group(1))} if m else set()


def lds_dma_hazards(asm: str) -> list:
    """Direct-to-LDS buffer loads come from inline asm, which the compiler's
    hazard recognizer does not look into: a VALU instruction that writes one of
    the load's descriptor SGPRs needs five wait states before the load reads
    it.  Returns a description of every load in `asm` (device assembly)
    without them."""
    lines = [l.strip() for l in asm.splitlines()]
    found, kernel = [], "?"
    for idx, line in enumerate(lines):
        if re.match(r"^_Z\S+:", line):
            kernel = line[:-1]
        if "buffer_load_dword" not in line or " lds" not in line:
            continue
        desc = _sgprs(line.split(",")[1].strip())
        ws, j = 0, idx - 1
        while j >= 0 and ws < 5:
            prev = lines[j]
            j -= 1
            if not prev or prev.startswith((";", ".")) or prev.endswith(":"):
                continue
            op = prev.split()[0]
            if op == "s_nop":
                ws += int(prev.split()[1], 0) + 1
                continue
            if op.startswith("v_") and _sgprs(prev.split()[1].rstrip(",")) & desc:
                found.append(f"{kernel}: '{prev}' {ws} wait states before '{line}'")
                break
            ws += 1
    return found


def build(verbose: bool = False) -> str:
    hipcc = _hipcc()
    os.makedirs(BUILD, exist_ok=True)
    jobs = []
    for src in HIP_SOURCES:
        path = os.path.join(CSRC, src)
        if not os.path.exists(path):
            continue
        obj = os.path.join(BUILD, src + ".o")
        jobs.append([hipcc, *COMMON, *DEVICE, "-x", "hip", "-c", path, "-o", obj])
    for src in CXX_SOURCES:
        obj = os.path.join(BUILD, src + ".o")
        jobs.append([hipcc, *COMMON, "-x", "c++", "-D__HIP_PLATFORM_AMD__",
                     f"-I{ROCM}/include", "-c", os.path.join(CSRC, src), "-o", obj])
    objs = [j[-1] for j in jobs]
    # device assembly of every HIP source, checked for unprotected loads
    asm_jobs = []
    for src in HIP_SOURCES:
        path = os.path.join(CSRC, src)
        if os.path.exists(path):
            asm_jobs.append([hipcc, *COMMON, *DEVICE, "--cuda-device-only", "-S", "-x", "hip", path,
                             "-o", os.path.join(BUILD, src + ".s")])
    with cf.ThreadPoolExecutor(max_workers=min(8, len(jobs) + len(asm_jobs))) as ex:
        for out in ex.map(_run, jobs + asm_jobs):
            if verbose and out.strip():
                print(out)
    hazards = []
    for j in asm_jobs:
        with open(j[-1]) as f:
            hazards += lds_dma_hazards(f.read())
    if hazards:
        raise RuntimeError("direct-to-LDS loads without the SGPR wait states:\n" + "\n".join(hazards))
    tmp = LIB + ".tmp"
    _run([hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp])
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
