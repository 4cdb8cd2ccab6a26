"""Build the HIP library in-tree: generator -> generated cores -> liballegro_tp.so.

Steps (every call rebuilds everything):
  1. g++ compiles the C++ coupling-table builder into the generator and runs it,
     writing csrc/generated/tp_cores.inc (straight-line contraction cores);
  2. g++ compiles the builder for the library (host code, -fPIC);
  3. hipcc compiles the kernels and the C ABI for gfx950 (the tensor product,
     then the layer around it), with packed-fp32 instruction selection disabled;
  4. hipcc links liballegro_tp.so next to this file, and builds bench.py's
     streaming probes (libstream_probe.so, not part of the ABI).
The per-kernel register / scratch report of step 3 is written to
_build/resource_usage.txt; a kernel that spills to scratch fails the build.
"""

from __future__ import annotations

import os
import re
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
GEN = os.path.join(CSRC, "generated")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "liballegro_tp.so")
PROBE_LIB = os.path.join(PKG, "libstream_probe.so")  # bench.py's streaming probes, outside the ABI
ARCH = "gfx950"
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
HIP_SOURCES = ("allegro_tp.hip", "allegro_layer.hip")  # tensor product; the layer around it
HIP_FLAGS = ["--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-I", os.path.join(ROOT, "include"), "-I", CSRC]


def _run(cmd, **kw):
    res = subprocess.run(cmd, capture_output=True, text=True, **kw)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("build step failed: " + " ".join(cmd[:3]) + " ...")
    return res


def _check_resources(report: str) -> str:
    """Summarise hipcc's kernel-resource-usage remarks; refuse scratch spills."""
    rows, current, bad = {}, None, []
    for ln in report.splitlines():
        m = re.search(r"remark: Function Name: (\S+)", ln)
        if m:
            current = m.group(1)
            rows[current] = {}
            continue
        m = re.search(r"remark:\s+([A-Za-z][A-Za-z ]*?)(?: \[[^\]]*\])?: (\S+) \[-Rpass", ln)
        if m and current:
            rows[current][m.group(1)] = m.group(2)
    out = []
    for name, kv in sorted(rows.items()):
        if kv.get("ScratchSize", "0") != "0" or kv.get("VGPRs Spill", "0") != "0":
            bad.append(name)
        out.append(f"{name} VGPRs={kv.get('VGPRs')} AGPRs={kv.get('AGPRs')} SGPRs={kv.get('TotalSGPRs')} "
                   f"scratch={kv.get('ScratchSize')} occupancy={kv.get('Occupancy')} lds={kv.get('LDS Size')}")
    if not rows:
        raise RuntimeError("no kernel resource report from hipcc")
    return "\n".join(out) + "\n", bad


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    os.makedirs(GEN, exist_ok=True)
    gen_exe = os.path.join(BUILD, "gen_kernels")
    _run(["g++", "-O2", "-std=c++17", os.path.join(CSRC, "gen_kernels.cpp"), os.path.join(CSRC, "cg_builder.cpp"),
          "-o", gen_exe])
    _run([gen_exe, os.path.join(GEN, "tp_cores.inc")])
    cg_obj = os.path.join(BUILD, "cg_builder.o")
    _run(["g++", "-O2", "-std=c++17", "-fPIC", "-c", os.path.join(CSRC, "cg_builder.cpp"), "-o", cg_obj])
    objs, report = [], ""
    for src in HIP_SOURCES:
        obj = os.path.join(BUILD, src.replace(".hip", ".o"))
        res = _run([HIPCC, *HIP_FLAGS, "-Rpass-analysis=kernel-resource-usage", "-c", os.path.join(CSRC, src),
                    "-o", obj])
        objs.append(obj)
        report += res.stderr
    summary, spills = _check_resources(report)
    with open(os.path.join(BUILD, "resource_usage.txt"), "w") as f:
        f.write(summary)
    if spills:
        raise RuntimeError("kernels use scratch memory (see _build/resource_usage.txt): " + ", ".join(spills))
    tmp = LIB + ".tmp"
    _run([HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", *objs, cg_obj, "-o", tmp])
    os.replace(tmp, LIB)
    tmp = PROBE_LIB + ".tmp"
    _run([HIPCC, *HIP_FLAGS, "-shared", os.path.join(CSRC, "stream_probe.hip"), "-o", tmp])
    os.replace(tmp, PROBE_LIB)
    if verbose:
        print(summary)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
