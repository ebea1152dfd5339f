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


# VALU instructions whose second operand is an SGPR destination (VOP3b
# carry-out / condition outputs); the first operand of any VALU instruction
# is its destination.
_VOP3B_SDST = re.compile(r"^v_(?:add_co|sub_co|subrev_co|addc_co|subb_co|subbrev_co)_u32"
                         r"|^v_div_scale_f(?:32|64)|^v_mad_(?:u64_u32|i64_i32)")
_BRANCH = re.compile(r"^s_(?:cbranch_\w+|branch)\s+(\S+)")
_NO_FALLTHROUGH = ("s_branch", "s_endpgm", "s_setpc_b64")


def _operands(line: str) -> list:
    parts = line.split(None, 1)
    return [t.strip() for t in parts[1].split(",")] if len(parts) > 1 else []


def _valu_sgpr_dests(line: str) -> set:
    op = line.split()[0]
    ops = _operands(line)
    out = _sgprs(ops[0]) if ops else set()
    if _VOP3B_SDST.match(op) and len(ops) > 1:
        out |= _sgprs(ops[1])
    return out


def lds_dma_hazards(asm: str) -> list:
    """Direct-to-LDS buffer loads come from inline asm, which the compiler's
    hazard recognizer does not look into.  Two hazards are checked:
    * a VALU instruction that writes one of the load's descriptor SGPRs (as
      its destination, or as the carry / condition output of a VOP3b form)
      needs five wait states before the load reads it;
    * an instruction that writes M0 needs one wait state before the load.
    Wait states are counted backwards along every path into the load: through
    a label into each branch that targets it (loop back-edges included) and
    into the fall-through predecessor, with one wait state per instruction
    and N + 1 per s_nop N.  The loads take their LDS address from M0, which
    the asm sets itself: in a function that holds such loads, an M0 write
    by compiler-generated code (outside the asm blocks) is a violation too,
    since it could fall between an M0 set-up and its loads.  Returns a
    description of every violation found in `asm` (device assembly)."""
    lines = [l.strip() for l in asm.splitlines()]
    preds = {}
    for i, l in enumerate(lines):
        m = _BRANCH.match(l)
        if m:
            preds.setdefault(m.group(1), []).append(i)
    found, kernel = [], "?"
    # compiler-generated M0 writes per function, and whether it has loads
    in_asm, m0_writes, has_dma = False, {}, set()
    for line in lines:
        if re.match(r"^_Z\S+:", line):
            kernel = line[:-1]
        if line.startswith(";;#ASMSTART"):
            in_asm = True
        elif line.startswith(";;#ASMEND"):
            in_asm = False
        elif "buffer_load_dword" in line and " lds" in line:
            has_dma.add(kernel)
        elif not in_asm and line[:1].isalpha() and _operands(line)[:1] == ["m0"]:
            m0_writes.setdefault(kernel, []).append(line)
    for k in sorted(has_dma):
        for w in m0_writes.get(k, []):
            found.append(f"{k}: compiler-generated M0 write '{w}' in a function with direct-to-LDS loads")
    kernel = "?"
    for idx, line in enumerate(lines):
        if re.match(r"^_Z\S+:", line):
            kernel = line[:-1]
        if "buffer_load_dword" not in line or " lds" not in line:
            continue
        desc = _sgprs(_operands(line)[1])
        # (line index, wait states so far, reached by a jump from that line)
        stack, seen = [(idx - 1, 0, False)], set()
        while stack:
            j, ws, jumped = stack.pop()
            while j >= 0 and ws < 5:
                if (j, ws, jumped) in seen:
                    break
                seen.add((j, ws, jumped))
                prev = lines[j]
                if prev.endswith(":"):
                    if not prev.startswith("."):
                        break  # function entry: no predecessor
                    stack.extend((b, ws, True) for b in preds.get(prev[:-1], []))
                    j -= 1
                    continue
                if not prev or prev.startswith((";", ".")):
                    j -= 1
                    continue
                op = prev.split()[0]
                if op in _NO_FALLTHROUGH and not jumped:
                    break  # control does not fall through into the code below
                jumped = False
                if op == "s_nop":
                    ws += int(prev.split()[1], 0) + 1
                    j -= 1
                    continue
                ops = _operands(prev)
                if ws < 1 and ops and ops[0] == "m0":
                    found.append(f"{kernel}: '{prev}' writes M0 {ws} wait states before '{line}'")
                if op.startswith("v_") and _valu_sgpr_dests(prev) & desc:
                    found.append(f"{kernel}: '{prev}' {ws} wait states before '{line}'")
                ws += 1
                j -= 1
    return sorted(set(found))


def _vgprs(tok: str) -> set:
    m = re.match(r"v\[(\d+):(\d+)\]", tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.match(r"v(\d+)$", tok)
    return {int(m.group(1))} if m else set()


def asm_valu_mfma_hazards(asm: str, need: int = 2) -> list:
    """A VALU instruction written in inline asm (the GEMM core's in-place
    sign flips of MFMA operand fragments) is invisible to the compiler's
    hazard recognizer, which would otherwise separate a VALU write of a VGPR
    from an MFMA that reads it by `need` wait states.  Following the
    fall-through path from each such write, with one wait state per
    instruction and N + 1 per s_nop N, an MFMA that reads the written VGPR
    (any source operand) before `need` wait states is a violation, and so is
    reaching a label or a branch first (the scan does not follow control
    flow).  Returns a description of every violation in `asm`."""
    lines = [l.strip() for l in asm.splitlines()]
    found, kernel, in_asm = [], "?", False
    for idx, line in enumerate(lines):
        if re.match(r"^_Z\S+:", line):
            kernel = line[:-1]
        if line.startswith(";;#ASMSTART"):
            in_asm = True
            continue
        if line.startswith(";;#ASMEND"):
            in_asm = False
            continue
        if not in_asm or not line.startswith("v_") or line.startswith("v_mfma"):
            continue
        ops = _operands(line)
        dst = _vgprs(ops[0]) if ops else set()
        if not dst:
            continue
        ws, j = 0, idx + 1
        while ws < need and j < len(lines):
            nxt = lines[j]
            j += 1
            if not nxt or nxt.startswith(";") or (nxt.startswith(".") and not nxt.endswith(":")):
                continue
            if nxt.endswith(":") or _BRANCH.match(nxt) or nxt.split()[0] in _NO_FALLTHROUGH:
                found.append(f"{kernel}: '{line}' reaches '{nxt}' before {need} wait states")
                break
            op = nxt.split()[0]
            if op == "s_nop":
                ws += int(nxt.split()[1], 0) + 1
                continue
            if op.startswith("v_mfma"):
                srcs = set().union(*(_vgprs(t) for t in _operands(nxt)[1:]))
                if srcs & dst:
                    found.append(f"{kernel}: '{line}' {ws} wait states before '{nxt}'")
            ws += 1
    return sorted(set(found))


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
            asm = f.read()
        hazards += lds_dma_hazards(asm) + asm_valu_mfma_hazards(asm)
    if hazards:
        raise RuntimeError("inline asm without the wait states it needs:\n" + "\n".join(hazards))
    tmp = LIB + ".tmp"
    _run([hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp])
    os.replace(tmp, LIB)
    return LIB


def build_host_sanitized(out: str | None = None) -> str:
    """libattr with its C-ABI layer (api.cpp) compiled by g++ under
    AddressSanitizer and UndefinedBehaviorSanitizer, linked with the device
    objects of the last build().  Only the host argument checks, planning and
    layout arithmetic are instrumented (kernels are not).  Load it with g++'s
    libasan preloaded and the library path in ATTR_LIBRARY."""
    gxx = shutil.which("g++")
    if gxx is None:
        raise RuntimeError("g++ not found")
    out = out or os.path.join(BUILD, "libattr_hostsan.so")
    dev_objs = [os.path.join(BUILD, s + ".o") for s in HIP_SOURCES]
    missing = [o for o in dev_objs if not os.path.exists(o)]
    if missing:
        raise RuntimeError(f"device objects missing (run build() first): {missing}")
    san = ["-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=undefined",
           "-fno-omit-frame-pointer"]
    obj = out + ".api.o"
    _run([gxx, "-O1", "-g", "-fPIC", "-std=c++17", *san, "-D__HIP_PLATFORM_AMD__",
          f"-I{ROCM}/include", f"-I{INCLUDE}", f"-I{CSRC}", "-c", os.path.join(CSRC, "api.cpp"),
          "-o", obj])
    _run([gxx, "-shared", *san, obj, *dev_objs, f"-L{ROCM}/lib", "-lamdhip64",
          f"-Wl,-rpath,{ROCM}/lib", "-o", out])
    return out


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
