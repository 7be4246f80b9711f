"""Build libpcr.so (HIP for gfx950) in-tree.

    python -m paper_2603_23049_amd.build

Compiles every source under csrc/ with hipcc for gfx950 and links them into
paper_2603_23049_amd/libpcr.so. Packed-fp32 instructions are disabled for all
device code.

The build also checks a register budget the layer pipeline depends on: an
attention workgroup (two waves per SIMD) must leave room on every SIMD for one
wave of the host-link copy kernel, so that the next layer's KV keeps streaming
into the pool while a long attention occupies every compute unit.
"""
from __future__ import annotations

import glob
import os
import re
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libpcr.so")
ROOT = os.path.dirname(HERE)

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-function", "-I", os.path.join(ROOT, "include")]


VGPRS_PER_SIMD_LANE = 512      # gfx950 register file per SIMD lane (VGPR + AGPR)
VGPR_GRANULE = 8               # allocation granule
ATTN_WAVES_PER_SIMD = 2        # 8-wave attention workgroup on 4 SIMDs


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def _alloc(n: int) -> int:
    return -(-n // VGPR_GRANULE) * VGPR_GRANULE


def _vgprs(remarks: str) -> dict:
    """Kernel name -> VGPRs + AGPRs, from -Rpass-analysis=kernel-resource-usage output."""
    out, name = {}, None
    for line in remarks.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            name = m.group(1)
            out[name] = 0
            continue
        m = re.search(r"\b(VGPRs|AGPRs): (\d+)", line)
        if m and name:
            out[name] += int(m.group(2))
    return out


def check_register_budget(usage: dict) -> None:
    attn = [v for k, v in usage.items() if "prefill_attn_kernel" in k]
    copy = [v for k, v in usage.items() if "copy_blocks_kernel" in k]
    if not attn or not copy:
        raise RuntimeError("register budget: kernel resource usage not found in the compiler remarks")
    need = ATTN_WAVES_PER_SIMD * _alloc(max(attn)) + _alloc(max(copy))
    if need > VGPRS_PER_SIMD_LANE:
        raise RuntimeError(f"register budget: attention {max(attn)} VGPRs x {ATTN_WAVES_PER_SIMD} waves + copy "
                           f"kernel {max(copy)} VGPRs = {need} > {VGPRS_PER_SIMD_LANE} per SIMD; the copy "
                           "kernel could not run beside the attention")


def build(verbose: bool = False, jobs: int = 4) -> str:
    objs = []
    procs = []
    os.makedirs(os.path.join(HERE, "_build"), exist_ok=True)
    remarks = []

    def finish(p, c):
        _, err = p.communicate()
        remarks.append(err)
        if p.returncode != 0:
            sys.stderr.write(err)
            raise RuntimeError("compile failed: " + " ".join(c))
        if verbose:
            sys.stderr.write("".join(l + "\n" for l in err.splitlines() if "remark" not in l))

    for src in sources():
        obj = os.path.join(HERE, "_build", os.path.basename(src) + ".o")
        cmd = [HIPCC, *FLAGS, "-Rpass-analysis=kernel-resource-usage", "-c", src, "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((subprocess.Popen(cmd, stderr=subprocess.PIPE, text=True), cmd))
        objs.append(obj)
        if len(procs) >= jobs:
            finish(*procs.pop(0))
    for p, c in procs:
        finish(p, c)
    check_register_budget(_vgprs("\n".join(remarks)))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
    sys.exit(0)
