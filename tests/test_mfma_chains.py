"""The generated gfx950 code never hands an MFMA accumulator from one MFMA shape to
another (no GPU: the kernels are compiled to assembly here).

A dependent 16x16x16 bf16 MFMA issued one or two instructions after the 16x16x32 bf16 MFMA
that produced its accumulator input (SrcC) read two of the four accumulator rows before
they were written: outputs at tokens 32 + {0, 1, 4, 5, 8, 9, 12, 13} of a chunk changed from
call to call.  Across three builds of the sequence kernels the failing instances were
exactly those where the compiler placed that pair one or two instructions apart; with five
wait states in between it never showed.  The kernels therefore keep every accumulator
chain on one shape, and this test checks the generated code for any exception: for each
MFMA whose SrcC is the destination of an earlier MFMA of another shape, with no other
write to those registers in between, it fails.  The search follows the code in program
order through labels and branches (a loop's last product and the first one after the
loop are such a pair however far apart they are), so it may also pair instructions on
paths that never run one after the other; that errs on the safe side.
"""
import os
import re
import shutil
import subprocess
import tempfile
from concurrent.futures import ThreadPoolExecutor

import pytest

from paper_2607_02805_amd import build

MFMA_SRCS = ("bdlm_scan.hip", "bdlm_seq.hip", "bdlm_mask.hip")   # the sources with MFMAs


def _regs(tok):
    m = re.match(r"[va]\[(\d+):(\d+)\]", tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.match(r"[va](\d+)$", tok)
    return {int(m.group(1))} if m else set()


def mixed_shape_chains(asm: str):
    """(function, first MFMA, dependent MFMA) for every accumulator handed between shapes,
    in program order within a function (labels and branches do not end the search)."""
    found = []
    for block in re.split(r"\n(?=_Z\w+:)", asm):
        m = re.match(r"(_Z\w+):", block)
        if not m:
            continue
        lines = [l.strip() for l in block.splitlines()
                 if l.strip() and not l.strip().startswith((";", "."))]
        for k, line in enumerate(lines):
            if not line.startswith("v_mfma"):
                continue
            t = line.replace(",", " ").split()
            dst = _regs(t[1])
            for u in lines[k + 1:]:
                if u.startswith("s_endpgm"):
                    break
                if u.endswith(":") or ":" in u.split()[0]:
                    continue
                tu = u.replace(",", " ").split()
                if u.startswith("v_mfma"):
                    if _regs(tu[4]) == dst and tu[0] != t[0]:
                        found.append((m.group(1)[:60], line, u))
                    if _regs(tu[1]) & dst or _regs(tu[4]) & dst:
                        break
                elif len(tu) > 1 and _regs(tu[1]) & dst:
                    break          # another instruction rewrites the registers
    return found


def _compile_to_asm(src: str, out: str) -> None:
    cmd = [build.HIPCC, *build.HIP_FLAGS, f"-I{build.INCLUDE}", f"-I{build.CSRC}",
           "--cuda-device-only", "-S", os.path.join(build.CSRC, src), "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]


@pytest.fixture(scope="module")
def asm_texts():
    if not (os.path.exists(build.HIPCC) or shutil.which(build.HIPCC)):
        pytest.skip("hipcc not available")
    with tempfile.TemporaryDirectory() as d:
        outs = {s: os.path.join(d, s.replace(".hip", ".s")) for s in MFMA_SRCS}
        with ThreadPoolExecutor(max_workers=len(outs)) as ex:
            for f in [ex.submit(_compile_to_asm, s, o) for s, o in outs.items()]:
                f.result()
        yield {s: open(o).read() for s, o in outs.items()}


@pytest.mark.parametrize("src", MFMA_SRCS)
def test_no_accumulator_crosses_mfma_shapes(asm_texts, src):
    asm = asm_texts[src]
    assert "v_mfma" in asm
    assert mixed_shape_chains(asm) == []


def test_the_scan_finds_a_planted_chain():
    """A 32-deep MFMA followed by a 16-deep one on its result is reported; the same pair
    on another accumulator, or with the registers rewritten in between, is not."""
    head = "_ZN4bdlm1fEv:\n"
    bad = head + ("\tv_mfma_f32_16x16x32_bf16 v[4:7], v[8:11], v[12:15], v[4:7]\n"
                  "\ts_waitcnt lgkmcnt(0)\n"
                  "\tv_mfma_f32_16x16x16_bf16 v[4:7], v[16:17], v[18:19], v[4:7]\n")
    assert len(mixed_shape_chains(bad)) == 1
    other = bad.replace("v[18:19], v[4:7]", "v[18:19], v[20:23]")
    assert mixed_shape_chains(other) == []
    rewritten = bad.replace("\ts_waitcnt lgkmcnt(0)\n", "\tv_mul_f32_e32 v4, v4, v30\n")
    assert mixed_shape_chains(rewritten) == []
    # across a loop exit, with other work in between: still reported
    far = bad.replace("\ts_waitcnt lgkmcnt(0)\n",
                      "\ts_cbranch_vccnz .LBB0_1\n.LBB0_2:\n" + "\tv_exp_f32_e32 v40, v41\n" * 50)
    assert len(mixed_shape_chains(far)) == 1
