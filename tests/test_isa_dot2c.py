"""The bf16 forward sums its probabilities with v_dot2c_f32_bf16.  In the
compensation kernel that instruction gave wrong sums when its accumulators
were registers an in-flight MFMA was reading; the forward is safe as long as
no v_dot2c accumulator is ever an MFMA operand.  This test compiles the
forward for gfx950 (device assembly, the library's own flags) and checks that
property on the code the compiler produces, so a compiler change that
allocates differently fails here instead of giving wrong sums."""
import os
import re
import shutil
import subprocess

import pytest

from paper_2609_23153_amd import build as B

KERNEL = "_ZN2sa12_GLOBAL__N_115fwd_bf16_kernelENS0_6ParamsE"


def _regs(tok):
    m = re.fullmatch(r"([va])(\d+)", tok)
    if m:
        return {(m.group(1), int(m.group(2)))}
    m = re.fullmatch(r"([va])\[(\d+):(\d+)\]", tok)
    if m:
        return {(m.group(1), k) for k in range(int(m.group(2)), int(m.group(3)) + 1)}
    return set()


def _operands(line):
    return [t.strip() for t in line.split(None, 1)[1].split(",")]


def kernel_instructions(asm, sym):
    lines = asm.split("\n")
    start = next(i for i, l in enumerate(lines) if l.startswith(sym + ":"))
    end = next(i for i in range(start, len(lines)) if "s_endpgm" in lines[i])
    return [l.split(";")[0].strip() for l in lines[start + 1:end]
            if l.strip() and not l.strip().startswith((";", ".")) and not l.rstrip().endswith(":")]


def dot2c_mfma_overlap(instrs):
    """(number of v_dot2c, accumulator registers that some MFMA reads or writes)."""
    acc, mfma = set(), set()
    n = 0
    for l in instrs:
        if l.startswith("v_dot2c"):
            n += 1
            acc |= _regs(_operands(l)[0])
        elif l.startswith("v_mfma"):
            for t in _operands(l)[:4]:
                mfma |= _regs(t)
    return n, acc & mfma


def test_scanner_sees_an_overlap():
    # the scanner itself: an accumulator that an MFMA reads is reported
    instrs = ["v_mfma_f32_32x32x16_bf16 a[0:15], v[4:7], v[8:11], a[0:15]",
              "v_dot2c_f32_bf16_e32 v9, v1, v2",
              "v_dot2c_f32_bf16_e32 v20, v1, v2"]
    n, bad = dot2c_mfma_overlap(instrs)
    assert n == 2 and bad == {("v", 9)}


@pytest.mark.skipif(not os.path.exists(B.HIPCC) and shutil.which("hipcc") is None,
                    reason="hipcc not available")
def test_fwd_bf16_dot2c_accumulators_are_never_mfma_operands(tmp_path):
    out = tmp_path / "fwd_bf16.s"
    cmd = [B.HIPCC, *B.FLAGS, "--cuda-device-only", "-S",
           os.path.join(B.CSRC, "fwd_bf16.hip"), "-o", str(out)]
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    assert r.returncode == 0, r.stdout
    instrs = kernel_instructions(out.read_text(), KERNEL)
    n, bad = dot2c_mfma_overlap(instrs)
    assert n > 0, "the forward no longer uses v_dot2c: drop this test"
    assert not bad, f"v_dot2c accumulators also used as MFMA operands: {sorted(bad)}"
