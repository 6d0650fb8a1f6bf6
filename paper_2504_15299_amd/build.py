"""Build libd2moe.so in-tree with hipcc for gfx950.

Every HIP source is compiled to an object file (in parallel) and linked into
``paper_2504_15299_amd/libd2moe.so``.  Packed fp32 VALU instructions are
disabled for all device code; the MWQ pack kernel is also compiled without
floating-point contraction because its integer codes must match the CPU
definition bit for bit.

The build also fails if any MFMA in the device assembly writes registers
that overlap its own source operands: multi-pass MFMAs read their sources
while they write, and the compiler does not always keep a 4-register result
apart from them (the decode kernels pin their operands to prevent it).

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
    _check_mfma(src)
    return obj


_REG = re.compile(r"([va])\[(\d+):(\d+)\]|([va])(\d+)$")


def _reg_range(tok: str):
    m = _REG.match(tok)
    if not m:
        return None
    if m.group(1):
        return m.group(1), int(m.group(2)), int(m.group(3))
    return m.group(4), int(m.group(5)), int(m.group(5))


def mfma_overlaps(asm: str) -> list[str]:
    """MFMA instructions whose destination overlaps srcA, srcB, a scale
    operand, or srcC other than exactly (in-place accumulation is allowed)."""
    bad = []
    for line in asm.splitlines():
        line = line.strip()
        if not line.startswith("v_mfma"):
            continue
        ops = [o.strip().split()[0] for o in line.split(None, 1)[1].split(",")]
        rs = [_reg_range(o) for o in ops]
        d = rs[0]
        srcs = rs[1:3] + (rs[4:6] if "scale" in line.split()[0] else [])
        if rs[3] != d:
            srcs.append(rs[3])
        for r in srcs:
            if d and r and d[0] == r[0] and not (d[2] < r[1] or r[2] < d[1]):
                bad.append(line)
                break
    return bad


def _check_mfma(src: str) -> None:
    cmd = [_hipcc(), *COMMON, *EXTRA.get(src, []), "--cuda-device-only", "-S", "-o", "-",
           os.path.join(CSRC, src)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc -S failed for {src}:\n{r.stderr}")
    bad = mfma_overlaps(r.stdout)
    if bad:
        raise RuntimeError(f"{src}: {len(bad)} MFMAs write over their own operands, e.g. {bad[0]}")


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
