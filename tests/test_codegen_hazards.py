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

Wait states are counted as issued instructions, ``s_nop N`` counting N + 1, along the
listing and along every branch into its target (a loop's back edge).
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


def parse(asm_text):
    """The kernels of an assembly listing: {name: [entry]}, each entry ("label", name) or
    ("ins", op, operands, inside_inline_asm, text)."""
    kernels, cur, in_asm = {}, None, False
    for line in asm_text.splitlines():
        s = line.strip()
        m = re.match(r"^(_Z\S+):", s)
        if m:
            cur, in_asm = [], False
            kernels[m.group(1)] = cur
            continue
        if cur is None:
            continue
        if s.startswith(";;#ASMSTART"):
            in_asm = True
            continue
        if s.startswith(";;#ASMEND"):
            in_asm = False
            continue
        m = re.match(r"^(\.?L\w+):", s)
        if m:
            cur.append(("label", m.group(1)))
            continue
        if not s or s.startswith(";") or s.startswith("."):
            continue
        parts = s.replace(",", " ").split()
        cur.append(("ins", parts[0], parts, in_asm, s))
    return kernels


class Window:
    """The last MFMA_TO_ACC_READ issue slots: VGPRs written by VALU and AGPRs written by an
    inline-assembly MFMA in each."""

    def __init__(self, valu=None, mfma=None):
        self.valu, self.mfma = list(valu or []), list(mfma or [])

    def copy(self):
        return Window(self.valu, self.mfma)

    def push(self, vw, md, n=1):
        for _ in range(n):
            self.valu.append(vw)
            self.mfma.append(md)
        del self.valu[:-MFMA_TO_ACC_READ]
        del self.mfma[:-MFMA_TO_ACC_READ]


def step(win, op, parts, in_asm):
    """Issue one instruction after the slots in `win`; returns the rule it breaks, or None,
    and the number of issue slots it took."""
    if op.startswith("s_nop"):
        n = int(parts[1], 0) + 1 if len(parts) > 1 else 1
        win.push(set(), set(), n)
        return None, n
    if op.startswith("v_mfma"):
        rule = None
        if in_asm:
            srcs = _regs(parts[2], "v") | _regs(parts[3], "v")
            recent = set().union(*win.valu[-VALU_TO_MFMA:]) if win.valu else set()
            if srcs & recent:
                rule = "VALU write -> MFMA read"
            win.push(set(), _regs(parts[1], "a"))
        else:
            win.push(set(), set())
        return rule, 1
    if op.startswith("v_accvgpr_read"):
        rule = "MFMA write -> accvgpr read" if _regs(parts[2], "a") & set().union(*win.mfma) else None
        win.push(_regs(parts[1], "v"), set())
        return rule, 1
    if op.startswith("v_") and not op.startswith("v_cmp") and len(parts) > 1:
        win.push(_regs(parts[1], "v"), set())
        return None, 1
    win.push(set(), set())
    return None, 1


def scan(asm_text):
    """Return a list of (kernel, rule, instruction) violations: along the listing, and along
    every branch into its target (a loop's back edge carries the end of the loop body to the
    instructions after the loop head)."""
    bad = set()
    for kernel, entries in parse(asm_text).items():
        labels = {e[1]: i for i, e in enumerate(entries) if e[0] == "label"}
        win, edges = Window(), []
        for e in entries:
            if e[0] != "ins":
                continue
            _, op, parts, in_asm, text = e
            rule, _ = step(win, op, parts, in_asm)
            if rule:
                bad.add((kernel, rule, text))
            if op.startswith(("s_branch", "s_cbranch")) and len(parts) > 1 and parts[1] in labels:
                edges.append((labels[parts[1]], win.copy()))
        for start, w in edges:   # the slots right after each branch target, entered by the branch
            used = 0
            for e in entries[start:]:
                if used >= MFMA_TO_ACC_READ:
                    break
                if e[0] != "ins":
                    continue
                _, op, parts, in_asm, text = e
                rule, n = step(w, op, parts, in_asm)
                used += n
                if rule:
                    bad.add((kernel, rule, text))
    return sorted(bad)


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
    # a loop whose last VALU write feeds the inline MFMA at its head: only the back edge
    # shows it (the listing runs the write last and falls out of the loop)
    loop = """_Zk:
.LBB0_1:
\t;;#ASMSTART
\tv_mfma_f32_16x16x32_f16 a[0:3], v[2:5], v[8:11], a[0:3]
\t;;#ASMEND
\ts_nop 7
\ts_nop 7
\ts_nop 7
\tv_cvt_pk_f16_f32 v2, v6, v7
{gap}\ts_cbranch_scc1 .LBB0_1
\ts_endpgm
"""
    assert [r for _, r, _ in scan(loop.format(gap=""))] == ["VALU write -> MFMA read"]
    assert scan(loop.format(gap="\ts_nop 0\n")) == []


def test_inline_mfma_hazards_absent(gemm_asm):
    kernels = set(re.findall(r"^(_Z\S*gemm_il_kernel\S*):", gemm_asm, re.M))
    # expand; projection store and accumulate, each with bf16 weights widened per fragment
    # and with float16 weights used as read; each on four and on eight waves
    assert len(kernels) == 10, kernels
    bad = scan(gemm_asm)
    assert bad == [], "\n".join(f"{k[:60]}: {r}: {i}" for k, r, i in bad[:10])
