"""Build libmtgnn.so (the HIP kernels and the C ABI) for gfx950, in-tree.

Usage:  python -m paper_2608_16305_amd.build   (or __graft_entry__.build())
"""

import concurrent.futures
import glob
import os
import re
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libmtgnn.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# Packed fp32 instructions are disabled: hipcc would otherwise form v_pk_* fp32
# ops from ordinary float code.
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", INCLUDE, "-I", SRC]


# Kernels that read LDS filled by direct global-to-LDS loads through inline
# assembly must not spill vector registers: a spill could copy a register before
# its LDS data has arrived.  The build fails if one of them does.  (Scalar
# registers spilled into vector-register lanes hold no LDS data.)
NO_SPILL = ("k_gemm_rs", "k_dw_rs", "k_dw_os")


def _spilling_kernels(remarks: str) -> list:
    """Names of kernels whose resource-usage remarks report a spill (NO_SPILL kernels) or any use of
    scratch memory (every kernel: private arrays that are indexed at run time land there, and
    each access is then a memory round trip)."""
    bad, name = [], None
    for line in remarks.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            name = m.group(1)
            continue
        m = re.search(r"VGPRs Spill: (\d+)", line)
        if m and name and int(m.group(1)) > 0 and any(k in name for k in NO_SPILL):
            bad.append(name)
        m = re.search(r"ScratchSize \[bytes/lane\]: (\d+)", line)
        if m and name and int(m.group(1)) > 0:
            bad.append(name)
    return bad


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    cmd = [HIPCC] + FLAGS + ["-Rpass-analysis=kernel-resource-usage", "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{r.stderr}")
    bad = _spilling_kernels(r.stderr)
    if bad:
        raise RuntimeError(f"{src}: kernels spill or use scratch memory: {sorted(set(bad))}")
    return obj


def build(jobs: int = 8) -> str:
    os.makedirs(BUILD, exist_ok=True)
    sources = sorted(glob.glob(os.path.join(SRC, "*.hip")))
    with concurrent.futures.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(_compile, sources))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(int(sys.argv[1]) if len(sys.argv) > 1 else 8))
