"""Static audit of the gfx950 kernels' machine code (CPU only).

Compiles the matrix-core kernels with the library's flags and checks what
the performance design relies on:
- no scratch (register spills) in any attention kernel;
- no register-file copies between VGPRs and AGPRs inside the kernels (every
  accumulator is a plain VGPR; a copy per tile would double the VALU work);
- no compiler-inserted wait for the direct-to-LDS loads right before an LDS
  read (the loads are issued through inline assembly precisely so that the
  next tile's loads stay in flight while the current tile is read).
If a code change makes the compiler spill, copy or serialize, this fails
here instead of showing up only as a slowdown on the GPU.
"""
import os
import re
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))



def _compile_to_asm(name):
    from paper_2606_01143_amd.build import COMMON_FLAGS, HIPCC
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    src = os.path.join(ROOT, "paper_2606_01143_amd", "csrc", name)
    out = os.path.join(tempfile.mkdtemp(prefix="spr_isa_"), "k.s")
    flags = [f for f in COMMON_FLAGS if f != "-fPIC"]
    r = subprocess.run([HIPCC, *flags, "--cuda-device-only", "-S", src, "-o", out],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    with open(out) as f:
        text = f.read()
    shutil.rmtree(os.path.dirname(out), ignore_errors=True)
    return text


def _functions(text, pattern):
    funcs = {}
    for m in re.finditer(r"^(_ZN3spr\w*" + pattern + r"\w*):", text, re.M):
        end = text.find(".Lfunc_end", m.end())
        funcs[m.group(1)] = [l.strip() for l in text[m.end():end].split("\n")
                             if l.strip() and not l.strip().startswith(";")]
    return funcs


@pytest.mark.parametrize("src,pattern", [("kernels_bf16_bwd.hip", "bwd_bf16_kernel"),
                                         ("kernels_bf16_bwd.hip", "bwd_kv_wide_kernel"),
                                         ("kernels_bf16_fwd.hip", "fwd_bf16_kernel"),
                                         ("kernels_bf16_fwd.hip", "fwd_wide_kernel")])
def test_kernels_do_not_spill_copy_or_serialize(src, pattern):
    funcs = _functions(_compile_to_asm(src), pattern)
    assert funcs, f"{pattern} not found in the assembly"
    for name, lines in funcs.items():
        assert any(l.startswith("v_mfma") for l in lines), f"{name}: no matrix instructions"
        spills = [l for l in lines if l.startswith("scratch_")]
        assert not spills, f"{name}: scratch spills: {spills[:5]}"
        copies = [l for l in lines if l.startswith("v_accvgpr_")]
        assert not copies, f"{name}: VGPR/AGPR copies: {copies[:5]}"
        waits = [i for i, l in enumerate(lines[:-1])
                 if l.startswith("s_waitcnt") and "vmcnt(0)" in l and lines[i + 1].startswith("ds_read")]
        assert not waits, f"{name}: vmcnt(0) right before an LDS read at lines {waits[:5]}"
