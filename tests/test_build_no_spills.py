"""Every kernel of libmsao.so keeps its vector registers: the gfx950 code
object built from csrc/ (the same hipcc flags as the library) reports no
VGPR spills and no scratch memory for any kernel. A VGPR spill turns into
scratch traffic in HBM and slows an HBM-bound pass (it happened once when a
store was added to the learned scoring instance, which runs at its
96-register limit). SGPR spills go to lanes of vector registers, not to
memory, and are allowed (the scoring pass keeps its per-channel activity
masks in scalar registers). Compiles on the CPU; no GPU needed."""
import os
import re
import subprocess

import pytest

from paper_2604_02945_amd import build as B

HIPCC = B.HIPCC
KERNEL_SOURCES = [s for s in B.SOURCES if s.endswith(".hip")]


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
@pytest.mark.parametrize("src", KERNEL_SOURCES, ids=os.path.basename)
def test_no_register_spills(src, tmp_path):
    flags = [f for f in B.FLAGS if f not in ("-fPIC", "-shared")]
    out = tmp_path / "k.s"
    r = subprocess.run([HIPCC, *flags, "--cuda-device-only", "-S", "-o", str(out), src],
                       capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-2000:]
    text = out.read_text()
    names = re.findall(r"^\s+\.name:\s+(\S+)$", text, re.M)
    kernels = [n for n in names if "_Z" in n and not n.endswith(".kd")]
    vspill = [int(v) for v in re.findall(r"\.vgpr_spill_count:\s+(\d+)", text)]
    sspill = [int(v) for v in re.findall(r"\.sgpr_spill_count:\s+(\d+)", text)]
    scratch = [int(v) for v in re.findall(r"\.private_segment_fixed_size:\s+(\d+)", text)]
    assert vspill and len(vspill) == len(sspill) == len(scratch)
    bad = [(k, v, p) for k, v, p in zip(kernels, vspill, scratch) if v or p]
    assert not bad, f"kernels that spill to memory (name, vgpr spills, scratch bytes): {bad}"
