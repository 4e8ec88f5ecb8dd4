"""Build libconduit.so (gfx950) in-tree with hipcc, and the benchmark's
matrix-core reference kernel as libconduit_ceiling.so.

    python -m paper_2609_05821_amd.build

Every HIP source is compiled for gfx950 only, with packed fp32 ops disabled
(the host pass warns that it does not know that feature; that is harmless).
"""
from __future__ import annotations

import concurrent.futures
import os
import re
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libconduit.so")
SOURCES = ["api.cpp", "attn.hip", "score.hip", "select.hip", "scatter.hip", "residual.hip", "static_ws.hip"]
CEILING_SRC = "ceiling.hip"  # measurement reference for bench.py, not part of the library
CEILING_LIB = os.path.join(PKG, "libconduit_ceiling.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", INCLUDE, "-I", CSRC]


# Per-kernel register, scratch and LDS figures from the compiler's remarks.
_REMARK = re.compile(r"remark:\s+(Function Name|VGPRs|AGPRs|ScratchSize \[bytes/lane\]|Occupancy \[waves/SIMD\]|"
                     r"LDS Size \[bytes/block\]):\s+(\S+)")


def resource_usage(stderr: str) -> dict:
    """{kernel symbol: {field: value}} from -Rpass-analysis=kernel-resource-usage."""
    out, cur = {}, None
    for key, val in _REMARK.findall(stderr):
        if key == "Function Name":
            cur = out.setdefault(val, {})
        elif cur is not None:
            cur[key.split(" ")[0]] = int(val)
    return out


def _compile(src: str) -> tuple:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *FLAGS, "-Rpass-analysis=kernel-resource-usage", "-x", "hip", "-c", os.path.join(CSRC, src),
           "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{res.stderr}")
    usage = {k: v for k, v in resource_usage(res.stderr).items() if "Occupancy" in v}  # kernels only
    # Per-lane scratch in a kernel means spilled registers or a kernel
    # parameter copied to private memory; every kernel here is written to
    # need none, so it is a build error.
    spills = {k: v["ScratchSize"] for k, v in usage.items() if v.get("ScratchSize", 0) > 0}
    if spills:
        raise RuntimeError(f"{src}: kernels using per-lane scratch memory: {spills}")
    return obj, usage


def build(verbose: bool = False) -> str:
    if not shutil.which(HIPCC) and not os.path.exists(HIPCC):
        raise RuntimeError("hipcc not found; the ROCm toolchain is required")
    os.makedirs(BUILD, exist_ok=True)
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(SOURCES) + 1)) as ex:
        done = list(ex.map(_compile, SOURCES + [CEILING_SRC]))
    objs = [o for o, _ in done]
    with open(os.path.join(BUILD, "resource_usage.txt"), "w") as f:
        for _, usage in done:
            for name, v in sorted(usage.items()):
                f.write(" ".join(f"{k}={v[k]}" for k in sorted(v)) + f" {name}\n")
    for lib, parts in ((LIB, objs[:-1]), (CEILING_LIB, objs[-1:])):
        tmp = lib + ".tmp"
        cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-Wl,--no-undefined", *parts, "-o", tmp]
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            raise RuntimeError(f"link failed:\n{res.stderr}")
        os.replace(tmp, lib)
        if verbose:
            print(f"built {lib}")
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
