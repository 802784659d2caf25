"""Build libselectinfer.so (HIP C++ for gfx950) in-tree with hipcc.

Usage: ``python -m paper_2607_18081_amd.build`` (or ``__graft_entry__.build()``).
Every call recompiles every source.
"""
from __future__ import annotations

import json
import os
import re
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libselectinfer.so")
USAGE = os.path.join(BUILD, "kernel_resource_usage.json")

ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CFLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # no packed-FP32 VALU instructions in any kernel
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # MFMAs accumulate in VGPRs: left to its heuristics the compiler keeps the accumulators in
    # AGPRs but feeds the MFMAs from VGPRs, copying every accumulator in and out around each
    # MFMA once the tiles use more than 256 registers in all
    "-mllvm", "-amdgpu-mfma-vgpr-form=1",
    "-I", INCLUDE, "-I", CSRC,
]


def sources() -> list[str]:
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hip"))


# the compiler's per-kernel resource remarks: kernel name, then (among others) its VGPR count
# and its scratch bytes per lane (register spills)
_REMARK = re.compile(r"remark:\s+(Function Name|VGPRs|ScratchSize \[bytes/lane\]): (\S+)")


def _compile(src: str) -> tuple[str, list]:
    obj = os.path.join(BUILD, os.path.basename(src)[:-4] + ".o")
    cmd = [HIPCC, *CFLAGS, "-Rpass-analysis=kernel-resource-usage", "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    usage, cur = [], None
    for key, val in _REMARK.findall(r.stderr):
        if key == "Function Name":
            cur = {"kernel": val, "source": os.path.basename(src)}
            usage.append(cur)
        elif cur is not None:
            cur["vgprs" if key == "VGPRs" else "scratch_bytes_per_lane"] = int(val)
    return obj, usage


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    srcs = sources()
    with ThreadPoolExecutor(min(8, len(srcs))) as ex:
        done = list(ex.map(_compile, srcs))
    objs = [o for o, _ in done]
    usage = [u for _, us in done for u in us]
    # every kernel instance's registers and scratch, for the no-spill check of the test suite
    with open(USAGE, "w") as f:
        json.dump(usage, f, indent=0)
    spills = [u["kernel"] for u in usage if u.get("scratch_bytes_per_lane", 0) > 0]
    if spills and verbose:
        print(f"warning: {len(spills)} kernel instance(s) use scratch: {spills[:4]}")
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "-shared", f"--offload-arch={ARCH}", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
