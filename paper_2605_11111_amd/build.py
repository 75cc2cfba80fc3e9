"""Build libshardconv.so (HIP, gfx950) in-tree with hipcc.

    python -m paper_2605_11111_amd.build      # always recompiles

Each source is compiled to an object in parallel, then linked. The library
lands next to this file, where the binding loads it. The measurement aid
libshardprobe.so (csrc/probe, declared in include/shardprobe.h) is built beside
it; the shard path never loads it.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import re
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OBJ = os.path.join(ROOT, "_build", "obj")
LIB = os.path.join(HERE, "libshardconv.so")
PROBE_LIB = os.path.join(HERE, "libshardprobe.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]


# Per-source code generation options. The forward W-march kernel keeps its
# weight fragments in AGPRs for the kernel's lifetime; with the MFMA results in
# VGPRs (VGPR form) the register allocator no longer shuffles those fragments
# between AGPRs on every tile, and the epilogue reads the accumulators directly.
SRC_FLAGS = {
    "conv_fwd_rows.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
    # the attention step holds scores, probabilities and V^T fragments for VALU
    # work next to the MFMA operands; in AGPR form the allocator spills
    "attention.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
}


def _compile(src: str) -> str:
    obj = os.path.join(OBJ, os.path.basename(src) + ".o")
    cmd = [HIPCC, *FLAGS, *SRC_FLAGS.get(os.path.basename(src), []), "-Rpass-analysis=kernel-resource-usage",
           "-x", "hip", "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"hipcc failed on {src}")
    _check_no_scratch(src, r.stderr)
    return obj


def _check_no_scratch(src: str, remarks: str) -> None:
    """The kernels issue LDS reads through inline asm and wait for them with
    explicit counters; that is only sound while the destination registers stay
    registers. A kernel that spills to scratch could store such a register
    before its data has arrived, so the build refuses any scratch use."""
    name = None
    for line in remarks.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            name = m.group(1)
        m = re.search(r"ScratchSize \[bytes/lane\]: (\d+)", line)
        if m and int(m.group(1)) != 0:
            raise RuntimeError(f"{os.path.basename(src)}: kernel {name} uses {m.group(1)} bytes/lane of scratch")


def _link(objs, lib: str) -> None:
    tmp = lib + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"link of {os.path.basename(lib)} failed")
    os.replace(tmp, lib)


def build(verbose: bool = False) -> str:
    os.makedirs(OBJ, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.cpp")))
    probe_srcs = sorted(glob.glob(os.path.join(CSRC, "probe", "*.hip")))
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs) + len(probe_srcs))) as ex:
        objs = list(ex.map(_compile, srcs + probe_srcs))
    _link(objs[:len(srcs)], LIB)
    _link(objs[len(srcs):], PROBE_LIB)
    if verbose:
        print(f"built {LIB} and {os.path.basename(PROBE_LIB)}")
    return LIB


if __name__ == "__main__":
    build(verbose=True)
