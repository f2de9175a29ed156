"""Code-generation checks of the attention kernels (CPU: hipcc cross-compiles
for gfx950; nothing runs on a GPU).

* The kernels whose tile loads go through inline assembly (forward, dQ, the
  D = 64 dK/dV kernel and the one-block D = 128 dK/dV kernel) must not wait
  for outstanding vector memory operations (`s_waitcnt vmcnt`) right before a
  transposed LDS read:
  that wait is the one the builtin load made the compiler insert, for the
  next tile's prefetch in the middle of the current tile.
* Register budgets the launch shapes rely on: no spills in any attention
  kernel, and the one-block D = 64 forward and dQ kernels within 128 VGPRs
  (four waves per SIMD).
"""
import os
import re
import shutil
import subprocess

import pytest

from paper_2405_13226_amd import build as B

HIPCC = B.HIPCC

pytestmark = pytest.mark.skipif(not (os.path.exists(HIPCC) or shutil.which("hipcc")),
                                reason="hipcc not available")


def device_asm(src, tmp_path):
    out = tmp_path / (src + ".s")
    cmd = [HIPCC, *B.HIP_FLAGS, *B.HIP_SOURCE_FLAGS.get(src, []), "--cuda-device-only", "-S",
           "-o", str(out), os.path.join(B.CSRC, src)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    return out.read_text()


def kernel_body(asm, mangled_prefix):
    """Instruction lines of the first kernel whose symbol starts with the prefix."""
    m = re.search(r"^(" + re.escape(mangled_prefix) + r"\w*):", asm, re.M)
    assert m, mangled_prefix
    start = m.end()
    end = asm.index(".end_amdhsa_kernel", start)
    lines = []
    for ln in asm[start:end].splitlines():
        t = ln.strip()
        if not t or t.startswith(";") or t.startswith(".") or t.endswith(":"):
            continue
        lines.append(t)
    return m.group(1), lines


def kernel_resources(asm):
    """{symbol: (vgpr_count, vgpr_spill_count)} from the metadata."""
    out = {}
    for m in re.finditer(r"\.name:\s+(_Z\S+)\s*\n(?:.*\n)*?\s+\.vgpr_count:\s+(\d+)\s*\n"
                         r"\s+\.vgpr_spill_count:\s+(\d+)", asm):
        out[m.group(1)] = (int(m.group(2)), int(m.group(3)))
    return out


def waits_before_transposed_reads(lines):
    n = 0
    for prev, cur in zip(lines, lines[1:]):
        if cur.startswith("ds_read_b64_tr_b16") and prev.startswith("s_waitcnt") and "vmcnt" in prev:
            n += 1
    return n


@pytest.mark.parametrize("src, prefix", [
    ("dd_bwd.hip", "_ZN2dd12dkdv1_kernelILi64ELb0E"),
    ("dd_bwd.hip", "_ZN2dd12dkdv1_kernelILi64ELb1E"),
    ("dd_bwd.hip", "_ZN2dd9dq_kernelILi64ELb0E"),
    ("dd_bwd.hip", "_ZN2dd9dq_kernelILi64ELb1E"),
    ("dd_bwd.hip", "_ZN2dd9dq_kernelILi128ELb0E"),
    ("dd_dkdv.hip", "_ZN2dd11dkdv_kernelILi128ELb0E"),
    ("dd_fwd.hip", "_ZN2dd10fwd_kernelILi64ELb0ELb0E"),
    ("dd_fwd.hip", "_ZN2dd10fwd_kernelILi64ELb1ELb0E"),
    ("dd_fwd.hip", "_ZN2dd10fwd_kernelILi128ELb0ELb0E"),
    ("dd_fwd.hip", "_ZN2dd10fwd_kernelILi128ELb1ELb0E"),
])
def test_no_dma_wait_before_transposed_reads(src, prefix, tmp_path):
    asm = device_asm(src, tmp_path)
    sym, lines = kernel_body(asm, prefix)
    assert any(ln.startswith("ds_read_b64_tr_b16") for ln in lines), sym
    assert waits_before_transposed_reads(lines) == 0, sym


@pytest.mark.parametrize("src", ["dd_fwd.hip", "dd_bwd.hip", "dd_dkdv.hip", "dd_bwd_short.hip"])
def test_attention_kernels_do_not_spill(src, tmp_path):
    res = kernel_resources(device_asm(src, tmp_path))
    assert res, src
    spills = {k: v for k, v in res.items() if v[1] != 0}
    assert not spills, spills
    four_waves = {"dd_fwd.hip": "_ZN2dd10fwd_kernelILi64ELb0ELb0E",
                  "dd_bwd.hip": "_ZN2dd9dq_kernelILi64ELb0E"}
    if src in four_waves:
        sym = next(k for k in res if k.startswith(four_waves[src]))
        assert res[sym][0] <= 128, res[sym]
