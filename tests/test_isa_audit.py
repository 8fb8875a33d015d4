"""Static audit of the backward kernel's machine code (CPU only).

The key-outer role keeps its dK/dV accumulators in AGPRs through inline-asm
matrix instructions that the compiler cannot see into.  That is only safe if
nothing else touches those registers while the products are in flight: no
spill, no copy, no read between the first and the last of these
instructions.  This test compiles the kernel source for gfx950 with the
library's flags and checks exactly that, so a code change that makes the
compiler spill or copy the accumulators fails here instead of producing
wrong gradients on the GPU.
"""
import os
import re
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "paper_2606_01143_amd", "csrc", "kernels_bf16_bwd.hip")


def _compile_to_asm():
    from paper_2606_01143_amd.build import COMMON_FLAGS, HIPCC
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    out = os.path.join(tempfile.mkdtemp(prefix="spr_isa_"), "bwd.s")
    flags = [f for f in COMMON_FLAGS if f != "-fPIC"]
    r = subprocess.run([HIPCC, *flags, "--cuda-device-only", "-S", SRC, "-o", out],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    with open(out) as f:
        text = f.read()
    shutil.rmtree(os.path.dirname(out), ignore_errors=True)
    return text


def _functions(text):
    funcs = {}
    for m in re.finditer(r"^(_ZN3spr15bwd_bf16_kernel\w+):", text, re.M):
        end = text.find(".Lfunc_end", m.end())
        funcs[m.group(1)] = text[m.end():end]
    return funcs


AGPR = re.compile(r"\ba(\d+|\[\d+:\d+\])")
ASM_MFMA = re.compile(r"^\s*v_mfma_\w+\s+a\[")


def test_agpr_accumulators_are_untouched_inside_the_sweep():
    text = _compile_to_asm()
    funcs = _functions(text)
    assert funcs, "backward kernel not found in the assembly"
    for name, body in funcs.items():
        lines = [l for l in body.split("\n") if l.strip() and not l.strip().startswith(";")]
        idx = [i for i, l in enumerate(lines) if ASM_MFMA.match(l)]
        assert idx, f"{name}: no AGPR-accumulating products found"
        bad = [l.strip() for l in lines[idx[0]:idx[-1] + 1]
               if AGPR.search(l) and not ASM_MFMA.match(l)]
        assert not bad, f"{name}: AGPR accessed inside the sweep: {bad[:5]}"
        spills = [l.strip() for l in lines if l.strip().startswith("scratch_")]
        assert not spills, f"{name}: scratch spills: {spills[:5]}"
