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

It also fails if the registers of an untracked (inline-asm) activation load
are read or written by anything else before the load's covering wait: their
data arrives late, so such a use would see, or be overwritten by, stale
data (a decode build whose loop copied a pointer through such registers
faulted on the GPU).

The same holds for LDS reads issued as inline assembly: their registers may
not be touched before the lgkmcnt wait that covers them.

And it fails if an inline-asm block that writes SCC is followed by a read of
SCC with no write in between: the compiler does not always treat the asm as
a definition of SCC, and a stale carry in a 64-bit scalar address add made
a decode build read from an illegal address.

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
EXTRA = {"pack.hip": ["-ffp-contract=off"], "calib.hip": ["-ffp-contract=off"]}


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
    # the device-assembly checks compile the source a second time; run that
    # compilation alongside the object build
    with cf.ThreadPoolExecutor(1) as ex:
        checks = ex.submit(_check_mfma, src)
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
        spills = scratch_users(r.stderr)
        if spills:
            raise RuntimeError(f"{src}: kernels use scratch memory (register spills): {spills}")
        checks.result()
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


def _vregs(tok: str) -> set[int]:
    m = re.match(r"v\[(\d+):(\d+)\]", tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.match(r"v(\d+)$", tok)
    return {int(m.group(1))} if m else set()


def _basic_blocks(lines: list[str], asm_markers: bool = False) -> list[dict]:
    """Basic blocks of one function's assembly (split at labels and after
    branches) with their successor indices.  With `asm_markers`, the
    compiler's inline-asm delimiters are kept as the pseudo-instructions
    ASMSTART / ASMEND."""
    blocks, cur = [], {"name": "entry", "ins": []}
    for line in lines:
        s = line.strip()
        m = re.match(r"^(\.LBB\S+):", s)
        if m:
            blocks.append(cur)
            cur = {"name": m.group(1), "ins": []}
            continue
        if asm_markers and s.startswith((";;#ASMSTART", ";;#ASMEND")):
            cur["ins"].append("ASMSTART" if "START" in s else "ASMEND")
            continue
        if not s or s.startswith((";", ".")):
            continue
        cur["ins"].append(s)
        if s.split()[0].startswith(("s_cbranch", "s_branch")):
            blocks.append(cur)
            cur = {"name": None, "ins": []}
    blocks.append(cur)
    index = {b["name"]: i for i, b in enumerate(blocks) if b["name"]}
    for i, b in enumerate(blocks):
        succ, falls = [], True
        for x in b["ins"]:
            op = x.split()[0]
            if op in ("ASMSTART", "ASMEND"):
                continue
            if op == "s_branch":
                succ.append(index[x.split()[1]])
                falls = False
            elif op.startswith("s_cbranch"):
                succ.append(index[x.split()[1]])
            elif op in ("s_endpgm", "s_setpc_b64"):
                falls = False
        if falls and i + 1 < len(blocks):
            succ.append(i + 1)
        b["succ"] = succ
    return blocks


_VMEM_PREFIXES = ("global_", "buffer_", "flat_", "scratch_")


def untracked_load_hazards(asm: str) -> list[tuple[str, str, str]]:
    """The decode kernels issue their activation loads as inline assembly
    (global_load_dwordx4 under a narrowed EXEC), and so do the 4-wave GEMM
    kernels (their A operands, one step ahead): the compiler does not track
    them, and the data lands in the destination registers some time later,
    when an explicit vmcnt wait covers it.  A load counts as untracked when it
    sits inside an inline-asm block or right after an EXEC narrowing.  Vector-memory instructions of a wave
    complete in order, so a wait `s_waitcnt vmcnt(N)` covers the load once at
    most N vector-memory instructions were issued after it on the path taken.
    On every path from such a load, no instruction may read or write its
    destination registers before the MFMA that consumes them as its B operand
    (the intended first use) or a covering wait: not another load, tracked or
    not, that reads them (as its address), nor anything else the compiler put
    there.  A later load may write them: its data lands after this one's.  (That each consuming MFMA sits behind a covering
    wait is not proven here: the walk is not path-sensitive, and the branch
    flags the compiler keeps in scalar registers make infeasible paths that
    skip the waits.  The wait counts are derived next to the loops that place
    them and exercised by the parity tests.)  Returns (function, load,
    offending instruction) triples."""
    bad = []
    for fname, lines in _funcs(asm).items():
        blocks = _basic_blocks(lines, asm_markers=True)
        # each instruction parsed once: (text, kind, value, registers), kind
        # "wait" (value: its vmcnt, or None), "mfma" (registers: its B
        # operand; value: the registers it reads otherwise), or "ins"
        # (registers: what it reads, value: whether it is vector memory)
        parsed = []
        for b in blocks:
            pb = []
            for y in b["ins"]:
                if y in ("ASMSTART", "ASMEND"):
                    continue
                op = y.split()[0]
                if op == "s_waitcnt":
                    m = re.search(r"vmcnt\((\d+)\)", y)
                    pb.append((y, "wait", int(m.group(1)) if m else None, None))
                    continue
                operands = y.split(None, 1)[1] if " " in y else ""
                reads = set()
                rd_ops = operands
                if _is_vector_load(op):
                    rd_ops = operands.split(",", 1)[1] if "," in operands else ""
                for t in re.findall(r"v\[\d+:\d+\]|v\d+\b", rd_ops):
                    reads |= _vregs(t)
                if op.startswith("v_mfma"):
                    ops = [o.strip() for o in operands.split(",")]
                    pb.append((y, "mfma", reads, _vregs(ops[2].split()[0])))
                else:
                    pb.append((y, "ins", op.startswith(_VMEM_PREFIXES), reads))
            parsed.append(pb)
        for bi, b in enumerate(blocks):
            inside = False
            k = 0  # index of the next parsed instruction of this block
            for ii, x in enumerate(b["ins"]):
                if x in ("ASMSTART", "ASMEND"):
                    inside = x == "ASMSTART"
                    continue
                k += 1
                if not x.startswith("global_load_dwordx4"):
                    continue
                if not inside and not any("s_and_saveexec" in y
                                          for y in b["ins"][max(0, ii - 3):ii]):
                    continue
                dst = _vregs(x.split()[1].rstrip(","))
                stack, seen = [(bi, k, 0)], set()
                while stack:
                    cb, ci, after = stack.pop()
                    if (cb, ci, after) in seen:
                        continue
                    seen.add((cb, ci, after))
                    stop = False
                    for y, kind, val, regs in parsed[cb][ci:]:
                        if kind == "wait":
                            if val is not None and val <= after:
                                stop = True      # the load has landed
                                break
                            continue
                        if kind == "mfma":
                            if regs & dst:
                                stop = True      # the consuming MFMA
                                break
                            # a later load may write the same registers (its
                            # data lands after this load's: loads complete in
                            # order), but none may read them, e.g. as its
                            # address
                            if val & dst:
                                bad.append((fname, x, y))
                                stop = True
                                break
                            continue
                        if regs & dst:
                            bad.append((fname, x, y))
                            stop = True
                            break
                        if val:
                            after = min(after + 1, 64)
                    if not stop:
                        stack.extend((sb, 0, after) for sb in blocks[cb]["succ"])
    return bad


def _is_vector_load(op: str) -> bool:
    """A vector-memory load that writes VGPRs (its first operand)."""
    return op.startswith(("global_load", "buffer_load", "flat_load", "scratch_load")) and \
        "_lds" not in op


def asm_lds_read_hazards(asm: str) -> list[tuple[str, str, str]]:
    """LDS reads issued as inline assembly (the decode and GEMM kernels read
    their DMA rings that way, so that the compiler does not drain the DMA
    queue before them) are, to the compiler, complete when the asm statement
    ends; their data lands only at the following `s_waitcnt lgkmcnt(0)`.  On
    every path from such a read to that wait, no instruction may touch its
    destination registers (another batched LDS read may use other
    registers; its address must not be one of them).  Returns (function,
    read, offending instruction) triples."""
    bad = []
    for fname, lines in _funcs(asm).items():
        blocks = _basic_blocks(lines, asm_markers=True)
        for bi, b in enumerate(blocks):
            inside = False
            for ii, x in enumerate(b["ins"]):
                if x == "ASMSTART":
                    inside = True
                    continue
                if x == "ASMEND":
                    inside = False
                    continue
                if not (inside and x.startswith("ds_read")):
                    continue
                dst = _vregs(x.split()[1].rstrip(","))
                stack, seen = [(bi, ii + 1)], set()
                while stack:
                    cb, ci = stack.pop()
                    if (cb, ci) in seen:
                        continue
                    seen.add((cb, ci))
                    stop = False
                    for y in blocks[cb]["ins"][ci:]:
                        if y in ("ASMSTART", "ASMEND"):
                            continue
                        op = y.split()[0]
                        if op == "s_waitcnt" and "lgkmcnt(0)" in y:
                            stop = True
                            break
                        operands = y.split(None, 1)[1] if " " in y else ""
                        if op.startswith("ds_read"):
                            operands = operands.split(",", 1)[1] if "," in operands else ""
                        hit = set()
                        for t in re.findall(r"v\[\d+:\d+\]|v\d+\b", operands):
                            hit |= _vregs(t)
                        if hit & dst:
                            bad.append((fname, x, y))
                            stop = True
                            break
                    if not stop:
                        stack.extend((sb, 0) for sb in blocks[cb]["succ"])
    return bad


_SCC_READERS = ("s_addc_u32", "s_subb_u32", "s_cselect_", "s_cbranch_scc", "s_cmov_", "s_cmovk_")
_SCC_WRITERS = ("s_add_", "s_sub_", "s_addc_", "s_subb_", "s_min_", "s_max_", "s_and_", "s_or_",
                "s_xor_", "s_andn2_", "s_orn2_", "s_nand_", "s_nor_", "s_xnor_", "s_lshl", "s_lshr",
                "s_ashr", "s_bfe_", "s_cmp_", "s_cmpk_", "s_bitcmp", "s_abs_", "s_not_", "s_absdiff")


def _funcs(asm: str) -> dict[str, list[str]]:
    funcs, name = {}, None
    for line in asm.splitlines():
        m = re.match(r"^(_Z\S+):", line)
        if m:
            name = m.group(1)
            funcs[name] = []
        elif name:
            funcs[name].append(line)
    return funcs


def scc_clobber_hazards(asm: str) -> list[tuple[str, str]]:
    """Inline-asm blocks that write SCC (s_and_saveexec, scalar arithmetic)
    after which, on some path, SCC is read before anything writes it again:
    the compiler kept a value in SCC across the asm (for instance the carry
    of a 64-bit scalar add), and the asm replaced it.  Returns (function,
    reading instruction) pairs."""
    bad = []
    for fname, lines in _funcs(asm).items():
        blocks = _basic_blocks(lines, asm_markers=True)
        for bi, b in enumerate(blocks):
            inside, writes = False, False
            for ii, x in enumerate(b["ins"]):
                if x == "ASMSTART":
                    inside, writes = True, False
                    continue
                if x == "ASMEND":
                    inside = False
                    if not writes:
                        continue
                    stack, seen = [(bi, ii + 1)], set()
                    while stack:
                        cb, ci = stack.pop()
                        if (cb, ci) in seen:
                            continue
                        seen.add((cb, ci))
                        stop = False
                        for y in blocks[cb]["ins"][ci:]:
                            if y in ("ASMSTART", "ASMEND"):
                                continue
                            op = y.split()[0]
                            if op.startswith(_SCC_READERS):
                                bad.append((fname, y))
                                stop = True
                                break
                            if op.startswith(_SCC_WRITERS) or "_saveexec_" in op:
                                stop = True
                                break
                        if not stop:
                            stack.extend((sb, 0) for sb in blocks[cb]["succ"])
                    continue
                if inside:
                    op = x.split()[0]
                    if op.startswith(_SCC_WRITERS) or "_saveexec_" in op:
                        writes = True
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
    sc = scc_clobber_hazards(r.stdout)
    if sc:
        raise RuntimeError(f"{src}: {len(sc)} reads of SCC that an inline-asm block overwrote, "
                           f"e.g. {sc[0]}")
    lz = asm_lds_read_hazards(r.stdout)
    if lz:
        raise RuntimeError(f"{src}: {len(lz)} inline-asm LDS reads whose registers are used before "
                           f"their lgkmcnt wait, e.g. {lz[0]}")
    hz = untracked_load_hazards(r.stdout)
    if hz:
        raise RuntimeError(f"{src}: {len(hz)} untracked activation loads whose registers are used "
                           f"before their covering wait, e.g. {hz[0]}")


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
