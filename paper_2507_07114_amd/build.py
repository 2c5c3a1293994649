"""Build liblossy.so (the HIP library behind include/lossy.h) and
libhbmprobe.so (the bandwidth probes behind include/hbm_probe.h) for gfx950.

Usage: python -m paper_2507_07114_amd.build   (or build() from Python).
The libraries are written next to this file so they travel with the source
tree.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(ROOT, "_build")
LIB_PATH = os.path.join(PKG, "liblossy.so")
PROBE_LIB_PATH = os.path.join(PKG, "libhbmprobe.so")

ARCH = "gfx950"
# -ffp-contract=off: every fused multiply-add in the kernels is explicit, so
# the fused step and the stage-by-stage entry points round identically.
# -packed-fp32-ops: keep the compiler from emitting packed fp32 VALU forms.
COMMON = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden",
    "-ffp-contract=off", "-Wall", "-Wextra", "-Wno-unused-result",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"-I{INCLUDE}", f"-I{CSRC}",
]
SOURCES = ["kernels.hip", "api.cpp"]
PROBE_SOURCES = ["probe.hip"]


def _hipcc() -> str:
    cand = os.environ.get("HIPCC") or shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(cand):
        raise RuntimeError(f"hipcc not found (looked for {cand})")
    return cand


def _run(cmd):
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(line for line in res.stdout.splitlines()
                    if "packed-fp32-ops" not in line and "not a recognized feature" not in line)
    if res.returncode != 0:
        raise RuntimeError(f"command failed ({res.returncode}): {' '.join(cmd)}\n{out}")
    return out


def _compile_jobs(hipcc, sources):
    objs, cmds = [], []
    for src in sources:
        obj = os.path.join(BUILD_DIR, os.path.splitext(src)[0] + ".o")
        objs.append(obj)
        cmds.append([hipcc, *COMMON, "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj])
    return objs, cmds


def _link(hipcc, objs, path):
    tmp = path + ".tmp"
    out = _run([hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp])
    os.replace(tmp, path)
    return out


def build(verbose: bool = False) -> str:
    """Compile every source for gfx950 and link liblossy.so and
    libhbmprobe.so; returns the path of liblossy.so."""
    hipcc = _hipcc()
    os.makedirs(BUILD_DIR, exist_ok=True)
    objs, cmds = _compile_jobs(hipcc, SOURCES)
    pobjs, pcmds = _compile_jobs(hipcc, PROBE_SOURCES)
    with ThreadPoolExecutor(max_workers=len(cmds) + len(pcmds)) as ex:
        outs = list(ex.map(_run, cmds + pcmds))
    outs.append(_link(hipcc, objs, LIB_PATH))
    outs.append(_link(hipcc, pobjs, PROBE_LIB_PATH))
    if verbose:
        for o in outs:
            if o.strip():
                print(o)
    return LIB_PATH


if __name__ == "__main__":
    path = build(verbose=True)
    print(path)
    sys.exit(0)
