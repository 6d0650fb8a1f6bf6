"""Build libd2moe.so in-tree with hipcc for gfx950.

Every HIP source is compiled to an object file (in parallel) and linked into
``paper_2504_15299_amd/libd2moe.so``.  Packed fp32 VALU instructions are
disabled for all device code; the MWQ pack kernel is also compiled without
floating-point contraction because its integer codes must match the CPU
definition bit for bit.

The build fails if any kernel needs per-lane scratch memory: the decode
kernels place their own vmcnt waits around the LDS DMA ring, which assume
that no other vector-memory traffic (such as register spills) is
interleaved, and in the other kernels a spill is a performance bug.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import re
import shutil
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(os.path.dirname(HERE), "include")
LIB = os.path.join(HERE, "libd2moe.so")
OBJ_DIR = os.path.join(HERE, "_build")

ARCH = "gfx950"
COMMON = ["-O3", "-fPIC", "-std=c++17", f"--offload-arch={ARCH}", "-I", INCLUDE,
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-Wno-unused-command-line-argument"]
EXTRA = {"pack.hip": ["-ffp-contract=off"]}


def _hipcc() -> str:
    p = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(p):
        raise RuntimeError("hipcc not found: the HIP library cannot be built")
    return p


def sources() -> list[str]:
    return sorted(f for f in os.listdir(CSRC) if f.endswith(".hip"))


def _compile(src: str) -> str:
    os.makedirs(OBJ_DIR, exist_ok=True)
    obj = os.path.join(OBJ_DIR, src.replace(".hip", ".o"))
    cmd = [_hipcc(), *COMMON, *EXTRA.get(src, []), "-Rpass-analysis=kernel-resource-usage",
           "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    spills = scratch_users(r.stderr)
    if spills:
        raise RuntimeError(f"{src}: kernels use scratch memory (register spills): {spills}")
    return obj


def scratch_users(remarks: str) -> dict[str, int]:
    """Kernels with a non-zero per-lane scratch size in the compiler's
    resource-usage remarks."""
    out, name = {}, None
    for line in remarks.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            name = m.group(1)
            continue
        m = re.search(r"ScratchSize \[bytes/lane\]: (\d+)", line)
        if m and name is not None and int(m.group(1)) > 0:
            out[name] = int(m.group(1))
    return out


def build(jobs: int | None = None) -> str:
    """Compile every HIP source and link the shared library.  Always
    recompiles (this is the 'does it build' check)."""
    srcs = sources()
    jobs = jobs or min(len(srcs), max(1, (os.cpu_count() or 4) // 2), 8)
    with cf.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(_compile, srcs))
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build())
