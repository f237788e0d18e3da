"""Builds the HIP library ``libstacklstm.so`` in-tree for gfx950 (hipcc, no JIT cache).

Every kernel's resource usage is read from the compiler's resource report, and the build
fails if a kernel that counts its own outstanding vector-memory operations (the wide
forward, the LDS-DMA ring GEMM, and the backward variants built with direct dA staging) uses
scratch memory: spill loads and stores share that counter, so a counted wait would no longer
wait for the loads it counts.

The device assembly of every source is kept (-save-temps) and scanned for one hazard the
compiler has been seen to miss: an MFMA chain at the end of a basic block whose results are
read at a branch target with fewer wait states than the compiler inserts for the same read
in straight-line code (the read then returns a stale accumulator). The build fails on one."""
from __future__ import annotations

import os
import re
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libstacklstm.so")
BUILD = os.path.join(HERE, "_build")
SOURCES = ["api.hip", "scan.hip", "gemm.hip", "recurrent_fwd.hip", "recurrent_fwd_pipe.hip", "recurrent_bwd.hip",
           "recurrent_fwd_wide.hip"]
# per-file flags: the wide forward keeps its U slice in AGPRs and its accumulators in VGPRs
EXTRA = {"recurrent_fwd_wide.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall",
         # packed fp32 instructions stay off: only scalar fp32 ALU code is generated
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Rpass-analysis=kernel-resource-usage"]


def bwd_direct_built(prec: int, nt: int, ks: int) -> bool:
    """The rule of rec_bwd_direct_built() in csrc/rec_config.h: backward variants that
    contain the direct-staging path (LDS DMA with counted waits)."""
    seg = ks * (32 if prec else 16) * (2 if prec else 4)
    occ = 2 if (prec == 1 and ks == 32) else 1
    return seg % 1024 == 0 and seg // 1024 <= 2 and occ == 1 and nt <= 4


def counted_waits(name: str) -> bool:
    """Kernels (mangled names) whose code counts outstanding vector-memory operations."""
    if name.startswith("_Z10k_fwd_wide") or name.startswith("_Z11k_gemm_ring"):
        return True
    # k_bwd<prec, NT, KS, OCC, GS>: the gate-split variants (GS = true) have no direct staging
    m = re.match(r"_Z5k_bwdILi(\d+)ELi(\d+)ELi(\d+)ELi(\d+)ELb([01])E", name)
    return bool(m) and m.group(5) == "0" and bwd_direct_built(int(m.group(1)), int(m.group(2)), int(m.group(3)))


def resource_report(text: str) -> dict:
    """{kernel: scratch bytes per lane} from hipcc's kernel-resource-usage remarks."""
    out, cur = {}, None
    for line in text.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            cur = m.group(1)
        m = re.search(r"ScratchSize \[bytes/lane\]: (\d+)", line)
        if m and cur:
            out[cur] = int(m.group(1))
    return out


# wait states between an MFMA and a read of its result that hipcc inserts in straight-line code
MFMA_WAITS = {"v_mfma_f32_16x16x4_f32": 10, "v_mfma_f32_16x16x32_bf16": 8}


def _regs(tok: str) -> set:
    m = re.fullmatch(r"([av])\[(\d+):(\d+)\]", tok)
    if m:
        return {(m.group(1), i) for i in range(int(m.group(2)), int(m.group(3)) + 1)}
    m = re.fullmatch(r"([av])(\d+)", tok)
    return {(m.group(1), int(m.group(2)))} if m else set()


def _split(line: str):
    parts = line.split(None, 1)
    if not parts:
        return "", []
    return parts[0], ([t.strip() for t in parts[1].split(",")] if len(parts) > 1 else [])


def _wait_states(line: str) -> int:
    op, args = _split(line)
    return int(args[0], 0) + 1 if op == "s_nop" else 1


def mfma_branch_hazards(asm: str) -> list:
    """Reads of MFMA results at a branch target with too few wait states since the MFMA.

    For every branch whose block ends with an MFMA (no other branch in between), the wait
    states from that MFMA to the branch are added to those from the target label up to the
    first instruction that reads the MFMA's destination registers (following fall-through,
    stopping at the next branch or MFMA); a total below MFMA_WAITS is reported."""
    lines = [ln.split(";")[0].strip() for ln in asm.splitlines()]
    labels = {ln[:-1]: i for i, ln in enumerate(lines) if re.fullmatch(r"\.?LBB\w+:", ln)}
    out, fn = [], "?"
    for i, ln in enumerate(lines):
        if re.fullmatch(r"_Z\w+:", ln):
            fn = ln[:-1]
        m = re.match(r"(s_cbranch_\w+|s_branch)\s+(\.LBB\w+)", ln)
        if not m or m.group(2) not in labels:
            continue
        w, dst, need = 1, None, 0
        for t in reversed(lines[max(0, i - 32):i]):
            if not t or t.endswith(":") or t.startswith(".") or t.startswith(";"):
                continue
            if t.startswith("v_mfma"):
                op, args = _split(t)
                dst, need = _regs(args[0]), MFMA_WAITS.get(op, 19)
                break
            if t.startswith(("s_cbranch", "s_branch", "s_setpc", "s_endpgm")):
                break
            w += _wait_states(t)
        if not dst:
            continue
        for t in lines[labels[m.group(2)] + 1:labels[m.group(2)] + 64]:
            if not t or t.endswith(":") or t.startswith("."):
                continue
            op, args = _split(t)
            if op.startswith("v_mfma") or op.startswith(("s_cbranch", "s_branch", "s_endpgm")) or w >= need:
                break
            if set().union(*[_regs(a) for a in args[1:]]) & dst:
                out.append(f"{fn}: {op} at {m.group(2)} reads an MFMA result after {w} wait states (needs {need})")
                break
            w += _wait_states(t)
    return out


def _compile(src: str):
    obj = os.path.join(BUILD, src.replace(".hip", ".o"))
    cmd = [HIPCC, *FLAGS, *EXTRA.get(src, []), "-save-temps", "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True, cwd=BUILD)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"hipcc failed for {src}")
    stem = src[:-len(".hip")]
    for f in os.listdir(BUILD):   # keep the device assembly and the objects only
        if f.startswith(stem + "-") and not f.endswith("-gfx950.s") or f.startswith(src + "-"):
            os.remove(os.path.join(BUILD, f))
    with open(os.path.join(BUILD, f"{stem}-hip-amdgcn-amd-amdhsa-gfx950.s")) as fh:
        hazards = mfma_branch_hazards(fh.read())
    return obj, resource_report(r.stderr), hazards


def build(jobs: int | None = None) -> str:
    os.makedirs(BUILD, exist_ok=True)
    jobs = jobs or min(len(SOURCES), max(1, (os.cpu_count() or 4)))
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        res = list(ex.map(_compile, SOURCES))
    objs = [o for o, _, _ in res]
    bad = {k: v for _, rep, _ in res for k, v in rep.items() if v > 0 and counted_waits(k)}
    if bad:
        raise RuntimeError(f"kernels with counted memory waits use scratch (bytes/lane): {bad}")
    hazards = [h for _, _, hz in res for h in hz]
    if hazards:
        raise RuntimeError("MFMA results read too early after a branch:\n" + "\n".join(hazards[:20]))
    tmp = LIB + ".tmp"
    subprocess.check_call([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-Wl,-z,defs", "-o", tmp, *objs])
    os.replace(tmp, LIB)
    return LIB


def scratch_report() -> dict:
    """Scratch bytes per lane of every kernel (compiles every source again)."""
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        res = list(ex.map(_compile, SOURCES))
    return {k: v for _, rep, _ in res for k, v in rep.items()}


if __name__ == "__main__":
    print(build())
