"""Build libpi_attn.so (HIP, gfx950) in-tree with hipcc.

    python -m paper_2511_10696_amd.build          # or build() from Python

Each ``csrc/*.hip`` is compiled to an object under ``_build/`` (in parallel)
and linked into ``paper_2511_10696_amd/libpi_attn.so``.
"""
from __future__ import annotations

import glob
import os
import re
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD_DIR = os.path.join(ROOT, "_build")
LIB_PATH = os.path.join(PKG, "libpi_attn.so")
ARCH = "gfx950"

# Packed-FP32 VALU instructions are disabled for every kernel (hipcc would
# otherwise form them from float2-style code).  MFMA accumulators are kept in
# ordinary VGPRs (the softmax rescales them with VALU instructions; the AGPR
# form would copy them back and forth).
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
VGPR_FORM = ["-mllvm", "-amdgpu-mfma-vgpr-form"]
COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-Wall",
          "-I", os.path.join(ROOT, "include")] + DEVICE_FLAGS


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    path = os.path.join(rocm, "bin", "hipcc")
    return path if os.path.exists(path) else "hipcc"


def sources() -> list[str]:
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


# The compiler's per-kernel resource remarks; the build fails if any kernel
# needs private (scratch) memory, i.e. spills registers.
RESOURCE_REMARKS = ["-Rpass-analysis=kernel-resource-usage"]


def scratch_users(remarks: str) -> list[str]:
    """Kernels whose resource remark reports a nonzero ScratchSize."""
    users, name = [], None
    for line in remarks.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            name = m.group(1)
            continue
        m = re.search(r"ScratchSize \[bytes/lane\]: (\d+)", line)
        if m and int(m.group(1)) > 0:
            users.append(f"{name} ({m.group(1)} bytes/lane)")
    return users


def _compile(src: str) -> str:
    obj = os.path.join(BUILD_DIR, os.path.basename(src) + ".o")
    cmd = [hipcc(), *COMMON, *VGPR_FORM, *RESOURCE_REMARKS, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    spills = scratch_users(r.stderr)
    if spills:
        raise RuntimeError(f"{src}: kernels use scratch memory (register spills): " + ", ".join(spills))
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD_DIR, exist_ok=True)
    srcs = sources()
    with ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(_compile, srcs))
    tmp = LIB_PATH + ".tmp"
    cmd = [hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB_PATH)
    if verbose:
        print(f"built {LIB_PATH}")
    return LIB_PATH


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
