"""Every kernel of libmsao.so keeps its vector registers and its buffer
descriptors scalar, checked on the gfx950 code object built from csrc/ (the
same hipcc flags as the library). Compiles on the CPU; no GPU needed.

* No VGPR spills and no scratch memory for any kernel. A VGPR spill turns
  into scratch traffic in HBM and slows an HBM-bound pass (it happened once
  when a store was added to the learned scoring instance, which runs at its
  96-register limit). SGPR spills go to lanes of vector registers, not to
  memory, and are allowed (the scoring pass keeps its per-channel activity
  masks in scalar registers).
* No waterfall loops. A buffer load or store takes its descriptor in scalar
  registers; when the compiler holds a descriptor in vector registers (a
  wavefront index taken from threadIdx without readfirstlane, a clamp done
  with a vector med3), it wraps every such access in a loop of
  readfirstlanes, compares and exec-mask updates. That loop once stood
  around every row load of the SimHash pass and of the fused clip pass,
  where it added VALU work to kernels that overlap VALU with streaming.
"""
import os
import re
import subprocess

import pytest

from paper_2604_02945_amd import build as B

HIPCC = B.HIPCC
KERNEL_SOURCES = [s for s in B.SOURCES if s.endswith(".hip") and "__global__" in open(s).read()]


@pytest.fixture(scope="module", params=KERNEL_SOURCES, ids=os.path.basename)
def asm(request, tmp_path_factory):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not installed")
    flags = [f for f in B.FLAGS if f not in ("-fPIC", "-shared")]
    out = tmp_path_factory.mktemp("asm") / "k.s"
    r = subprocess.run([HIPCC, *flags, "--cuda-device-only", "-S", "-o", str(out), request.param],
                       capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-2000:]
    return out.read_text()


def test_no_register_spills(asm):
    names = re.findall(r"^\s+\.name:\s+(\S+)$", asm, re.M)
    kernels = [n for n in names if "_Z" in n and not n.endswith(".kd")]
    vspill = [int(v) for v in re.findall(r"\.vgpr_spill_count:\s+(\d+)", asm)]
    sspill = [int(v) for v in re.findall(r"\.sgpr_spill_count:\s+(\d+)", asm)]
    scratch = [int(v) for v in re.findall(r"\.private_segment_fixed_size:\s+(\d+)", asm)]
    assert vspill and len(vspill) == len(sspill) == len(scratch)
    bad = [(k, v, p) for k, v, p in zip(kernels, vspill, scratch) if v or p]
    assert not bad, f"kernels that spill to memory (name, vgpr spills, scratch bytes): {bad}"


def waterfall_loops(asm):
    """(function, loop label) of every loop that re-reads a vector operand
    lane by lane: a back edge taken while exec is non-zero to a short block
    that starts with a readfirstlane and holds an equality compare against it
    and an exec-mask save (a branch to an exit block laid out earlier is not
    one)."""
    found = []
    funcs = re.finditer(r"^(_Z\S+):[^\n]*\n(.*?)^\.Lfunc_end", asm, re.M | re.S)
    for f in funcs:
        body = f.group(2)
        for m in re.finditer(r"s_cbranch_execnz\s+(\.LBB\S+)", body):
            label = m.group(1)
            start = body.find(label + ":")
            if start < 0 or start > m.start():
                continue
            lines = [l.strip() for l in body[start:m.start()].split("\n")[1:]]
            insts = [l for l in lines if l and not l.startswith(";")]
            loop = "\n".join(insts)
            if (insts and insts[0].startswith("v_readfirstlane") and len(insts) <= 40
                    and re.search(r"v_cmp_eq_u(32|64)", loop) and "s_and_saveexec" in loop):
                found.append((f.group(1), label))
    return found


def test_no_waterfall_loops(asm):
    bad = waterfall_loops(asm)
    assert not bad, f"loads or stores with a per-lane descriptor (function, loop): {bad[:8]} ({len(bad)} loops)"


def test_the_waterfall_check_sees_one():
    """The check on a hand-written loop of the shape the compiler emits."""
    text = "\n".join([
        "_Zk:                                    ; @_Zk",
        "\ts_mov_b64 s[12:13], exec",
        ".LBB0_7:",
        "\tv_readfirstlane_b32 s8, v10",
        "\tv_readfirstlane_b32 s9, v11",
        "\tv_cmp_eq_u64_e64 s[0:1], s[8:9], v[10:11]",
        "\ts_and_saveexec_b64 s[0:1], s[0:1]",
        "\tbuffer_load_dwordx4 v[60:63], v9, s[8:11], 0 offen nt",
        "\ts_xor_b64 exec, exec, s[0:1]",
        "\ts_cbranch_execnz .LBB0_7",
        "\ts_endpgm",
        ".Lfunc_end0:",
    ])
    assert waterfall_loops(text) == [("_Zk", ".LBB0_7")]
    assert waterfall_loops(text.replace("v_readfirstlane_b32", "s_mov_b32")) == []
