"""Build libbdlm.so in-tree: HIP kernels for gfx950 with hipcc, the C ABI with g++.

Usage: ``python -m paper_2607_02805_amd.build``.  Always recompiles.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libbdlm.so")
PROBE_LIB = os.path.join(HERE, "libbdlm_probe.so")

ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# Packed-fp32 VALU ops are kept out of the device code; the host pass of hipcc
# warns that it does not know the feature, which is harmless.
HIP_FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-munsafe-fp-atomics",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-Wall", "-Wno-unused-function"]


def _run(cmd: list[str]) -> None:
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"build step failed: {' '.join(cmd)}")
    noise = "is not a recognized feature for this target"
    for line in (r.stdout + r.stderr).splitlines():
        if line.strip() and noise not in line:
            sys.stderr.write(line + "\n")


HIP_SRCS = ("bdlm_scan.hip", "bdlm_seq.hip", "bdlm_mask.hip", "bdlm_conv.hip", "bdlm_norm.hip",
            "bdlm_scratch.hip")


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    cmds, objs = [], []
    for src in HIP_SRCS:
        obj = os.path.join(BUILD, src.replace(".hip", ".o"))
        cmds.append([HIPCC, *HIP_FLAGS, f"-I{INCLUDE}", f"-I{CSRC}", "-c",
                     os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    a_obj = os.path.join(BUILD, "bdlm_api.o")
    cmds.append(["g++", "-O2", "-std=c++17", "-fPIC", "-Wall", "-Wextra", f"-I{INCLUDE}",
                 f"-I{CSRC}", "-c", os.path.join(CSRC, "bdlm_api.cpp"), "-o", a_obj])
    # the translation units are independent: compile them side by side
    with ThreadPoolExecutor(max_workers=min(len(cmds), os.cpu_count() or 1)) as ex:
        for f in [ex.submit(_run, c) for c in cmds]:
            f.result()
    tmp = LIB + ".tmp"
    _run([HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp, *objs, a_obj])
    os.replace(tmp, LIB)
    # the benchmark's streaming probe: a library of its own, outside the product ABI
    ptmp = PROBE_LIB + ".tmp"
    _run([HIPCC, *HIP_FLAGS, "-shared", "-o", ptmp, os.path.join(CSRC, "bdlm_probe.hip")])
    os.replace(ptmp, PROBE_LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build(verbose=True)
