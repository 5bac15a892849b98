"""Device-code checks of the grouped GEMM kernels (CPU only: hipcc cross-compiles gfx950).

The large-tile kernel issues its MFMAs through inline assembly (to pin the accumulators to
AGPRs), and the compiler's hazard recognizer does not look inside inline assembly. Two
rules therefore have to hold by construction of the code, and this test reads the
generated assembly to check them:

* a VALU write of a VGPR is at least two wait states ahead of an inline-assembly MFMA that
  reads it as its A or B operand (the compiler puts ``s_nop 1`` there for its own MFMAs;
  a missing gap made the projection read stale fragments);
* an inline-assembly MFMA's accumulator is not read by ``v_accvgpr_read`` within 18 wait
  states (more than the 16-pass MFMA latency).

Wait states are counted as issued instructions, ``s_nop N`` counting N + 1.
"""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_01024_amd", "csrc")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"

VALU_TO_MFMA = 2
MFMA_TO_ACC_READ = 18


def _regs(tok, prefix):
    m = re.match(prefix + r"\[(\d+):(\d+)\]$", tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.match(prefix + r"(\d+)$", tok)
    return {int(m.group(1))} if m else set()


def scan(asm_text):
    """Return a list of (kernel, rule, instruction) violations."""
    bad = []
    kernel, in_asm = None, False
    valu_writes = []   # per issue slot: VGPRs written by VALU
    mfma_dsts = []     # per issue slot: AGPRs written by an inline-assembly MFMA
    def push(vw, md, n=1):
        for _ in range(n):
            valu_writes.append(vw)
            mfma_dsts.append(md)
        del valu_writes[:-MFMA_TO_ACC_READ]
        del mfma_dsts[:-MFMA_TO_ACC_READ]
    for line in asm_text.splitlines():
        s = line.strip()
        m = re.match(r"^(_Z\S+):", s)
        if m:
            kernel, in_asm = m.group(1), False
            valu_writes.clear()
            mfma_dsts.clear()
            continue
        if s.startswith(";;#ASMSTART"):
            in_asm = True
            continue
        if s.startswith(";;#ASMEND"):
            in_asm = False
            continue
        if not s or s.startswith(";") or s.startswith("."):
            continue
        parts = s.replace(",", " ").split()
        op = parts[0]
        if op.startswith("s_nop"):
            push(set(), set(), int(parts[1], 0) + 1 if len(parts) > 1 else 1)
            continue
        if op.startswith("v_mfma"):
            if in_asm:
                srcs = _regs(parts[2], "v") | _regs(parts[3], "v")
                recent = set().union(*valu_writes[-VALU_TO_MFMA:]) if valu_writes else set()
                if srcs & recent:
                    bad.append((kernel, "VALU write -> MFMA read", s))
                push(set(), _regs(parts[1], "a"))
            else:
                push(set(), set())
            continue
        if op.startswith("v_accvgpr_read"):
            src = _regs(parts[2], "a")
            if src & set().union(*mfma_dsts):
                bad.append((kernel, "MFMA write -> accvgpr read", s))
            push(_regs(parts[1], "v"), set())
            continue
        if op.startswith("v_") and not op.startswith("v_cmp") and len(parts) > 1:
            push(_regs(parts[1], "v"), set())
            continue
        push(set(), set())
    return bad


@pytest.fixture(scope="module")
def gemm_asm(tmp_path_factory):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    out = tmp_path_factory.mktemp("asm") / "gemm_bf16.s"
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature",
           "-Xclang", "-packed-fp32-ops", "-I", os.path.join(ROOT, "include"), "-I", CSRC, "-S",
           "--cuda-device-only", os.path.join(CSRC, "gemm_bf16.hip"), "-o", str(out)]
    subprocess.run(cmd, check=True, capture_output=True)
    return out.read_text()


def test_scanner_flags_planted_hazards():
    """The scanner itself: a VALU write right before an inline MFMA, and an early
    accumulator read, are reported; the same code with enough wait states is not."""
    bad = """_Zk:
\tv_cvt_pk_f16_f32 v2, v6, v7
\t;;#ASMSTART
\tv_mfma_f32_16x16x32_f16 a[0:3], v[2:5], v[8:11], a[0:3]
\t;;#ASMEND
\tv_accvgpr_read_b32 v20, a1
"""
    good = """_Zk:
\tv_cvt_pk_f16_f32 v2, v6, v7
\ts_nop 1
\t;;#ASMSTART
\tv_mfma_f32_16x16x32_f16 a[0:3], v[2:5], v[8:11], a[0:3]
\t;;#ASMEND
\ts_nop 7
\ts_nop 7
\ts_nop 7
\tv_accvgpr_read_b32 v20, a1
"""
    rules = sorted(r for _, r, _ in scan(bad))
    assert rules == ["MFMA write -> accvgpr read", "VALU write -> MFMA read"]
    assert scan(good) == []


def test_inline_mfma_hazards_absent(gemm_asm):
    kernels = set(re.findall(r"^(_Z\S*gemm_il_kernel\S*):", gemm_asm, re.M))
    assert len(kernels) == 3, kernels   # expand, projection store, projection accumulate
    bad = scan(gemm_asm)
    assert bad == [], "\n".join(f"{k[:60]}: {r}: {i}" for k, r, i in bad[:10])
