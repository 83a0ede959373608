"""Static check of the library's gfx950 machine code for the wave-level
hazards that hand-written assembly in the kernels could create and the
compiler cannot see through: a DPP instruction reading a VGPR within two
wait states of the VALU instruction that wrote it (the DPP butterflies and
lane max/min blocks are inline asm), and an LDS-DMA load
(global_load_lds_*) within one wait state of an SALU write of M0 (the
GEMMs' DMA blocks set M0 themselves).

The code objects are taken from the built libquarot.so (its .hip_fatbin
section, one offload bundle per source file) and disassembled with the
ROCm LLVM tools; nothing runs on a GPU.  Straight-line code is checked:
the scan restarts at every label, so a hazard whose two instructions sit
in different basic blocks would not be seen."""
import os
import re
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2404_00456_amd", "libquarot.so")
LLVM = "/opt/rocm/llvm/bin"
MAGIC = b"__CLANG_OFFLOAD_BUNDLE__"

pytestmark = pytest.mark.skipif(
    not (os.path.exists(LIB) and os.path.exists(os.path.join(LLVM, "llvm-objdump"))),
    reason="needs the built library and the ROCm LLVM tools")


def disassemble():
    """gfx950 disassembly of every code object in the library."""
    out = []
    with tempfile.TemporaryDirectory() as d:
        fb = os.path.join(d, "fatbin")
        subprocess.run(["objcopy", "-O", "binary", "--only-section=.hip_fatbin", LIB, fb],
                       check=True)
        data = open(fb, "rb").read()
        offs = [m.start() for m in re.finditer(re.escape(MAGIC), data)] + [len(data)]
        for i in range(len(offs) - 1):
            part = os.path.join(d, f"b{i}")
            with open(part, "wb") as f:
                f.write(data[offs[i]:offs[i + 1]])
            co = os.path.join(d, f"b{i}.co")
            subprocess.run([os.path.join(LLVM, "clang-offload-bundler"), "--unbundle",
                            "--type=o", f"--input={part}",
                            "--targets=hipv4-amdgcn-amd-amdhsa--gfx950", f"--output={co}"],
                           check=True)
            res = subprocess.run([os.path.join(LLVM, "llvm-objdump"), "-d", "--mcpu=gfx950",
                                  co], capture_output=True, text=True, check=True)
            out.append(res.stdout)
    return out


REG = re.compile(r"\bv\[(\d+):(\d+)\]|\bv(\d+)\b")


def vregs(text):
    regs = set()
    for m in REG.finditer(text):
        if m.group(3) is not None:
            regs.add(int(m.group(3)))
        else:
            regs.update(range(int(m.group(1)), int(m.group(2)) + 1))
    return regs


def parse(line):
    """(mnemonic, operand text) of an instruction line, or None."""
    code = line.split("//")[0].strip()
    if not code or code.endswith(":"):
        return None
    parts = code.split(None, 1)
    return parts[0], parts[1] if len(parts) > 1 else ""


DPP_CTL = ("quad_perm:", "row_shl:", "row_shr:", "row_ror:", "row_mirror", "row_half_mirror",
           "row_bcast", "wave_shl", "wave_shr", "wave_rol", "wave_ror", "row_share", "row_xmask")


def check(text):
    """Violations in one disassembly: (function, line, message)."""
    bad = []
    func = "?"
    recent = []  # (wait states since, mnemonic, vgprs written, writes m0)
    for raw in text.splitlines():
        s = raw.strip()
        m = re.match(r"^[0-9a-f]+ <(.+)>:$", s)
        if m:
            func, recent = m.group(1), []
            continue
        if s.endswith(":") or s.startswith("<"):
            recent = []  # a label: another path may enter here
            continue
        p = parse(raw)
        if p is None or p[0].startswith((".", "Disassembly")):
            continue
        mn, ops = p
        is_dpp = any(c in ops for c in DPP_CTL) or mn.endswith("_dpp")
        if is_dpp:
            # the DPP-read source is the first source operand
            fields = [f.strip() for f in ops.split(",")]
            src0 = vregs(fields[1]) if len(fields) > 1 else set()
            for waits, pmn, pregs, _ in recent:
                if waits < 2 and pmn.startswith("v_") and src0 & pregs:
                    bad.append((func, s, f"DPP reads v{sorted(src0 & pregs)} {waits} wait "
                                         f"state(s) after {pmn} wrote it"))
        if "_lds_" in mn and mn.startswith(("global_load", "buffer_load")):
            for waits, pmn, _, wm0 in recent:
                if wm0 and waits < 1:
                    bad.append((func, s, f"LDS DMA {waits} wait state(s) after {pmn} wrote m0"))
        # age the window: s_nop N gives N + 1 wait states, anything else one
        step = int(ops, 0) + 1 if mn == "s_nop" else 1
        recent = [(w + step, a, b, c) for (w, a, b, c) in recent if w + step < 8]
        if mn != "s_nop":
            fields = [f.strip() for f in ops.split(",")]
            dst = fields[0] if fields else ""
            writes_v = vregs(dst) if mn.startswith("v_") and not mn.startswith(
                ("v_cmp", "v_readlane", "v_readfirstlane")) else set()
            writes_m0 = mn.startswith("s_") and dst == "m0"
            recent.append((0, mn, writes_v, writes_m0))
    return bad


def test_no_dpp_or_m0_hazards():
    texts = disassemble()
    assert len(texts) >= 5  # one code object per source file with kernels
    ndpp = sum(t.count("_dpp") + t.count("quad_perm") for t in texts)
    nlds = sum(t.count("global_load_lds") for t in texts)
    assert ndpp > 100 and nlds > 10  # the checked patterns are present
    bad = [v for t in texts for v in check(t)]
    assert not bad, "\n".join(f"{f}: {l}: {m}" for f, l, m in bad[:20])


def test_checker_sees_a_planted_hazard():
    """The checker itself, on hand-written listings: a DPP read right after
    the write and an LDS DMA right after an M0 write are reported; with
    the wait states in place they are not."""
    good = """0000000000000000 <k>:
\tv_add_f32_e32 v4, v5, v6
\ts_nop 1
\tv_mov_b32_dpp v7, v4 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf
\ts_mov_b32 m0, s3
\ts_nop 0
\tglobal_load_lds_dwordx4 v2, off
"""
    bad = good.replace("\ts_nop 1\n", "").replace("\ts_nop 0\n", "")
    assert check(good) == []
    found = check(bad)
    assert len(found) == 2 and "DPP" in found[0][2] and "m0" in found[1][2]
