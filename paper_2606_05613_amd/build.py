"""Build libbkmoo.so (HIP for gfx950) in-tree with hipcc.

    python -m paper_2606_05613_amd.build

Every translation unit under csrc/ is compiled in parallel into _build/ and
linked into paper_2606_05613_amd/libbkmoo.so.  All device code is built with
packed-fp32 instruction selection disabled; the units holding the solvers
(the solve and exact-solve kernels and the cooperative kernel that embeds
them) and the conflict statistics additionally without floating-point
contraction, so their scalar expressions round as written.

After compiling, the generated gfx950 assembly is checked, and the build
fails on either finding:
  * a vector-memory store of more than 64 bits whose data registers an
    immediately following vector instruction overwrites (the store reads its
    data over two cycles and such an overwrite corrupts the stored value);
  * a cross-workgroup hand-off of either pipelined resolve kernel out of order:
    every publish point (an inline "s_waitcnt vmcnt(0)" marked "bkmoo
    publish") must be followed, in the same block, by the flag or counter
    update as its next vector-memory instruction, and every observe point
    (marked "bkmoo observe") must follow a poll loop with no vector-memory
    load between the loop's s_sleep and the point.
"""

from __future__ import annotations

import concurrent.futures
import glob
import os
import re
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libbkmoo.so")
ARCH = "gfx950"

SOURCES = ["api.hip", "schedule.hip", "gram.hip", "solve.hip", "solve_exact.hip", "combine.hip",
           "hybrid.hip", "refill.hip", "conflicts.hip", "slices.hip"]
EXTRA = {"solve.hip": ["-ffp-contract=off"], "solve_exact.hip": ["-ffp-contract=off"],
         "hybrid.hip": ["-ffp-contract=off"], "refill.hip": ["-ffp-contract=off"],
         "conflicts.hip": ["-ffp-contract=off"]}


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libbkmoo)")


def common_flags():
    return [f"--offload-arch={ARCH}", "-O3", "-fPIC", "-std=c++17",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-I", INCLUDE, "-I", CSRC]


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, src.replace(".hip", ".o"))
    cmd = [hipcc()] + common_flags() + EXTRA.get(src, []) + ["-save-temps=obj", "-c",
                                                             os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True, cwd=BUILD)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{r.stderr[-6000:]}")
    return obj


def _vgprs(op: str):
    m = re.match(r"v\[(\d+):(\d+)\]", op)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.match(r"v(\d+)$", op)
    return {int(m.group(1))} if m else set()


def store_data_overwrites(asm_path: str):
    """(line, store, next instruction) where a >64-bit vector store is
    followed directly by a vector instruction writing its data registers."""
    lines = [ln.split(";")[0].strip() for ln in open(asm_path)]
    found = []
    for i, ln in enumerate(lines):
        m = re.match(r"(buffer|global|flat|scratch)_store_(dwordx3|dwordx4|b96|b128)\s+(.*)", ln)
        if not m:
            continue
        ops = [o.strip() for o in m.group(3).split(",")]
        data = _vgprs(ops[0] if m.group(1) == "buffer" else ops[1])
        for nxt in lines[i + 1:i + 4]:
            if not nxt or nxt.startswith("."):
                continue
            w = re.match(r"v_\w+\s+([^,]+)", nxt)
            if w and _vgprs(w.group(1).strip()) & data:
                found.append((i + 1, ln, nxt))
            break
    return found


VMEM = re.compile(r"^\s*(global|buffer|flat|scratch)_(\w+)")
LABEL = re.compile(r"^[.\w$]+:")


def _kernels(lines, name_part):
    """(name, first line, end line) of each function whose symbol contains name_part."""
    out, cur = [], None
    for i, ln in enumerate(lines):
        m = re.match(r"^(_Z\S+):\s*(;.*)?$", ln)
        if m and name_part in m.group(1):
            cur = (m.group(1), i)
        elif cur and ln.startswith(".Lfunc_end"):
            out.append((cur[0], cur[1], i))
            cur = None
    return out


def handoff_order_violations(asm_path: str, kernel: str = "hybrid_kernel"):
    """(line, problem) for every hand-off of `kernel` that is out of order, or
    a kernel with no publish or no observe point at all."""
    lines = open(asm_path).read().splitlines()
    found = []
    for name, lo, hi in _kernels(lines, kernel):
        pubs = [i for i in range(lo, hi) if "bkmoo publish" in lines[i]]
        obss = [i for i in range(lo, hi) if "bkmoo observe" in lines[i]]
        if not pubs or not obss:
            found.append((lo + 1, f"{name}: no publish or no observe point"))
        for i in pubs:
            for j in range(i + 1, hi):
                ln = lines[j].split(";")[0].rstrip()
                if LABEL.match(ln):
                    found.append((i + 1, "a block starts between a publish point and its flag update"))
                    break
                m = VMEM.match(ln)
                if m:
                    op = m.group(1) + "_" + m.group(2)
                    if not (op == "global_atomic_add" or (op == "global_store_dword" and " sc1" in ln)):
                        found.append((i + 1, f"publish point followed by {op}, not the flag or counter"))
                    break
            else:
                found.append((i + 1, "publish point with no update after it"))
        for i in obss:
            for j in range(i - 1, lo, -1):
                ln = lines[j].split(";")[0].strip()
                if ln.startswith("s_sleep"):
                    break
                m = VMEM.match(ln)
                if m and "load" in m.group(2):
                    found.append((i + 1, f"{m.group(1)}_{m.group(2)} between a poll loop and an observe point"))
                    break
            else:
                found.append((i + 1, "observe point with no poll loop before it"))
    return found


def build(jobs: int = 8) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with concurrent.futures.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(_compile, SOURCES))
    bad = []
    for asm in glob.glob(os.path.join(BUILD, f"*-hip-amdgcn-amd-amdhsa-{ARCH}.s")):
        bad += [(os.path.basename(asm),) + h for h in store_data_overwrites(asm)]
    if bad:
        detail = "\n".join(f"{a}:{ln}: {st}  ->  {nx}" for a, ln, st, nx in bad[:20])
        raise RuntimeError(f"{len(bad)} store-data overwrite hazards in the generated code:\n{detail}")
    for unit, kernel in (("hybrid", "hybrid_kernel"), ("refill", "refill_kernel")):
        asm = os.path.join(BUILD, f"{unit}-hip-amdgcn-amd-amdhsa-{ARCH}.s")
        order = handoff_order_violations(asm, kernel)
        if order or not _kernels(open(asm).read().splitlines(), kernel):
            detail = "\n".join(f"{unit}.s:{ln}: {what}" for ln, what in order[:20]) or f"no {kernel} found"
            raise RuntimeError(f"cross-workgroup hand-off out of order in the generated code:\n{detail}")
    tmp = LIB + ".tmp"
    cmd = [hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr[-6000:]}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(int(sys.argv[1]) if len(sys.argv) > 1 else 8))
