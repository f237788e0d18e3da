"""Builds the HIP library ``libstacklstm.so`` in-tree for gfx950 (hipcc, no JIT cache).

Every kernel's resource usage is read from the compiler's resource report, and the build
fails if a kernel that counts its own outstanding vector-memory operations (the wide
forward, and the backward variants built with direct dA staging) uses scratch memory:
spill loads and stores share that counter, so a counted wait would no longer wait for the
loads it counts."""
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
    if name.startswith("_Z10k_fwd_wide"):
        return True
    m = re.match(r"_Z5k_bwdILi(\d+)ELi(\d+)ELi(\d+)ELi(\d+)E", name)
    return bool(m) and bwd_direct_built(int(m.group(1)), int(m.group(2)), int(m.group(3)))


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


def _compile(src: str):
    obj = os.path.join(BUILD, src.replace(".hip", ".o"))
    cmd = [HIPCC, *FLAGS, *EXTRA.get(src, []), "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"hipcc failed for {src}")
    return obj, resource_report(r.stderr)


def build(jobs: int | None = None) -> str:
    os.makedirs(BUILD, exist_ok=True)
    jobs = jobs or min(len(SOURCES), max(1, (os.cpu_count() or 4)))
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        res = list(ex.map(_compile, SOURCES))
    objs = [o for o, _ in res]
    bad = {k: v for _, rep in res for k, v in rep.items() if v > 0 and counted_waits(k)}
    if bad:
        raise RuntimeError(f"kernels with counted memory waits use scratch (bytes/lane): {bad}")
    tmp = LIB + ".tmp"
    subprocess.check_call([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-Wl,-z,defs", "-o", tmp, *objs])
    os.replace(tmp, LIB)
    return LIB


def scratch_report() -> dict:
    """Scratch bytes per lane of every kernel (compiles every source again)."""
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        res = list(ex.map(_compile, SOURCES))
    return {k: v for _, rep in res for k, v in rep.items()}


if __name__ == "__main__":
    print(build())
