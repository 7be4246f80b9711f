"""CPU: register use of the kernels, read from the compiler's resource report and
assembly for gfx950 (no GPU needed): no kernel spills, and the attention's tile loop
(four softmax / matrix phase pairs per iteration) holds every MFMA of its four tiles
with no scratch access and no SGPR reload in it."""
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2603_23049_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["-O3", "-std=c++17", "--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include")]


def _resources(src):
    cmd = [HIPCC, *FLAGS, "-c", os.path.join(CSRC, src), "-o", os.devnull, "-Rpass-analysis=kernel-resource-usage"]
    out = subprocess.run(cmd, capture_output=True, text=True, check=True).stderr
    res, cur = {}, None
    for line in out.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            cur = m.group(1)
            res[cur] = {}
            continue
        m = re.search(r"remark:\s+([A-Za-z ]+?)(?: \[[^\]]*\])?: (\d+)", line)
        if m and cur:
            res[cur][m.group(1).strip()] = int(m.group(2))
    return res


def _granule(v):
    return -(-v // 8) * 8


pytestmark = pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")


def test_no_kernel_spills():
    for src in ("attn.hip", "decode.hip", "kv_move.hip"):
        for name, r in _resources(src).items():
            assert r["VGPRs Spill"] == 0 and r["SGPRs Spill"] == 0 and r["ScratchSize"] == 0, (src, name, r)
    a128 = [v for k, v in _resources("attn.hip").items() if "prefill_attn_kernelILi128" in k]
    assert a128 and a128[0]["LDS Size"] <= 160 * 1024 and a128[0]["VGPRs"] <= 256


def test_attention_tile_loop_has_no_spill_traffic():
    """The loop that runs four (softmax, matrix) phase pairs per iteration holds every
    MFMA of four tiles; no scratch access and no SGPR reload (v_readlane) may sit in it."""
    out = subprocess.run([HIPCC, *FLAGS, "--cuda-device-only", "-S", os.path.join(CSRC, "attn.hip"), "-o", "-"],
                         capture_output=True, text=True, check=True).stdout
    start = out.index("prefill_attn_kernelILi128")
    body = out[start:out.index(".Lfunc_end", start)].split("\n")
    labels = {m.group(1): i for i, l in enumerate(body) if (m := re.match(r"^(\.LBB\d+_\d+):", l))}
    loops = []
    for i, l in enumerate(body):
        m = re.search(r"s_cbranch_\w+\s+(\.LBB\d+_\d+)\s*$|s_branch\s+(\.LBB\d+_\d+)\s*$", l)
        lab = m and (m.group(1) or m.group(2))
        if lab in labels and labels[lab] < i:
            loops.append(body[labels[lab]:i + 1])
    def count(lines, pat):
        return sum(1 for x in lines if re.search(pat, x))
    # four phase pairs: 4 x (32 products + 4 row sums) MFMAs, and nothing more
    hot = [lp for lp in loops if count(lp, r"v_mfma") == 4 * 36]
    assert hot, "tile loop with four phase pairs not found"
    for lp in hot:
        assert count(lp, r"scratch_") == 0 and count(lp, r"v_readlane|v_writelane") == 0
