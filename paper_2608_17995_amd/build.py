"""Build libavits.so for gfx950 with hipcc (in-tree, no torch involvement).

    python -m paper_2608_17995_amd.build
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
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libavits.so")
ARCH = "gfx950"

SOURCES = ("abi.hip", "score.hip", "select.hip", "relayout.hip", "gemm.hip", "attention.hip", "block.hip",
           "noise.hip")

CXXFLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-mcode-object-version=5",
    # Packed fp32 VALU ops are kept out of every kernel.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-result",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        raise RuntimeError("build failed:\n" + " ".join(cmd) + "\n" + r.stdout)
    return r.stdout


# Kernels that must compile without scratch: the GEMM's loads are
# asynchronous inline assembly (a spilled destination would be saved before
# the data lands); a spill in the attention or scoring tile loops costs more
# than half their speed; the selections keep their keys in registers.
NO_SCRATCH = {"gemm.hip": ("gemm_bf16",), "attention.hip": ("attn_bf16_kernel",),
              "score.hip": ("spatial_temporal_bf16", "finalize_select"), "select.hip": ("radix_select",)}
_USAGE = ["-Rpass-analysis=kernel-resource-usage"]


def _check_no_scratch(src: str, out: str) -> None:
    want = NO_SCRATCH[src]
    name = None
    for line in out.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            name = m.group(1)
            continue
        m = re.search(r"ScratchSize \[bytes/lane\]: (\d+)", line)
        if m and name and any(w in name for w in want) and int(m.group(1)) != 0:
            raise RuntimeError(f"{src}: {name} uses {m.group(1)} bytes of scratch per lane; it must build "
                               "without spills")


def build(verbose: bool = False, jobs: int | None = None) -> str:
    """Compile every HIP source for gfx950 and link libavits.so; returns its path."""
    os.makedirs(BUILD, exist_ok=True)
    cc = hipcc()
    objs = []
    cmds = []
    for src in SOURCES:
        obj = os.path.join(BUILD, src.replace(".hip", ".o"))
        objs.append(obj)
        extra = _USAGE if src in NO_SCRATCH else []
        cmds.append([cc, *CXXFLAGS, *extra, f"-I{INCLUDE}", f"-I{CSRC}", "-c", os.path.join(CSRC, src), "-o", obj])
    jobs = jobs or min(len(cmds), os.cpu_count() or 4, 8)
    with cf.ThreadPoolExecutor(jobs) as ex:
        for src, out in zip(SOURCES, ex.map(_run, cmds)):
            if src in NO_SCRATCH:
                _check_no_scratch(src, out)
            elif verbose and out.strip():
                print(out)
    tmp = LIB + ".tmp"
    _run([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs])
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
