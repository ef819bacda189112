"""Build libdcp.so in-tree with hipcc for gfx950.

``python -m paper_2608_07524_amd.build`` (or ``build()``) compiles every HIP
and C++ source under ``csrc/`` and links ``paper_2608_07524_amd/libdcp.so``.
It always recompiles: the build is the check that the sources compile.
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
LIB = os.path.join(PKG, "libdcp.so")
# measurement probe library (bench.py's counter calibration), not part of libdcp
PROBE_SOURCES = ["probe/dma_copy.hip", "probe/mfma_rate.hip"]
PROBE_LIB = os.path.join(PKG, "libdcp_probe.so")

SOURCES = ["attn_fwd.hip", "attn_bwd.hip", "layer.hip", "dcp_api.cpp", "dcp_error.cpp", "work_list.cpp", "dcp_plan.cpp",
           "layer_api.cpp", "noalloc.hip"]

# Packed fp32 vector ops stay disabled for device code (plain scalar fp32
# VALU only); the host pass reports the feature as unknown, which is benign.
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
COMMON_FLAGS = ["-O3", "-std=c++17", "-fPIC", "--offload-arch=gfx950", "-Wall", "-Wno-unused-function",
                "-I", INCLUDE, "-I", CSRC]


def _hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found; ROCm is required to build libdcp")


def _compile(hipcc: str, src: str, obj: str):
    cmd = [hipcc, *COMMON_FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
    if src.endswith(".hip"):
        cmd[1:1] = ["-x", "hip"]
        cmd += DEVICE_FLAGS
    res = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in res.stderr.splitlines() if "packed-fp32-ops" not in l)
    if res.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{err}")
    return err


def build(verbose: bool = False, out: str = LIB, build_dir: str = BUILD_DIR) -> str:
    """Compile every source and link ``out`` (the in-tree libdcp.so by default)."""
    hipcc = _hipcc()
    os.makedirs(build_dir, exist_ok=True)
    objs = [os.path.join(build_dir, os.path.splitext(s)[0] + ".o") for s in SOURCES]
    with ThreadPoolExecutor(max_workers=min(6, len(SOURCES))) as ex:
        logs = list(ex.map(lambda so: _compile(hipcc, so[0], so[1]), zip(SOURCES, objs)))
    if verbose:
        for s, log in zip(SOURCES, logs):
            if log.strip():
                print(f"--- {s}\n{log}", file=sys.stderr)
    tmp = out + ".tmp"
    cmd = [hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs, "-L/opt/rocm/lib", "-lrocblas",
           "-Wl,-rpath,/opt/rocm/lib"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{res.stderr}")
    os.replace(tmp, out)
    if out == LIB:
        build_probe(build_dir)
    return out


def build_probe(build_dir: str = BUILD_DIR) -> str:
    """The measurement probes bench.py loads (libdcp_probe.so)."""
    hipcc = _hipcc()
    os.makedirs(build_dir, exist_ok=True)
    objs = []
    for src in PROBE_SOURCES:
        obj = os.path.join(build_dir, os.path.basename(os.path.splitext(src)[0]) + ".o")
        _compile(hipcc, src, obj)
        objs.append(obj)
    tmp = PROBE_LIB + ".tmp"
    res = subprocess.run([hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs], capture_output=True,
                         text=True)
    if res.returncode != 0:
        raise RuntimeError(f"probe link failed\n{res.stderr}")
    os.replace(tmp, PROBE_LIB)
    return PROBE_LIB


if __name__ == "__main__":
    print(build(verbose=True))
