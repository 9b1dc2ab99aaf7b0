"""Constraints on the generated gfx950 code that the sources rely on (CPU).

The inline-assembly global-to-LDS copy (dma16_opaque in csrc/common.h) sets
M0, a register the compiler reserves and does not take as clobbered.  It is
correct only in kernels where the compiler itself emits no M0 use: this
test cross-compiles the sources to assembly and checks every kernel that
contains the copy.
"""
import os
import re
import shutil
import subprocess
import tempfile

import pytest

from paper_2606_07577_amd import build

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(os.path.dirname(HERE), "paper_2606_07577_amd", "csrc")


def _device_asm(src):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    with tempfile.TemporaryDirectory() as d:
        out = os.path.join(d, "k.s")
        cmd = [hipcc, *build.FLAGS, "--cuda-device-only", "-S", os.path.join(CSRC, src), "-o", out]
        res = subprocess.run(cmd, capture_output=True, text=True)
        assert res.returncode == 0, res.stderr[-2000:]
        return open(out).read()


def _kernels(asm):
    for m in re.finditer(r"^(_Z\w+):\s*(?:;.*)?$", asm, re.M):
        end = asm.find(".Lfunc_end", m.end())
        yield m.group(1), asm[m.end():end]


@pytest.mark.parametrize("src", ["redundancy.hip"])
def test_opaque_copies_share_no_m0_with_the_compiler(src):
    asm = _device_asm(src)
    checked = 0
    for name, body in _kernels(asm):
        inside, has_copy, stray = False, False, []
        for line in body.splitlines():
            t = line.strip()
            if t.startswith(";;#ASMSTART"):
                inside = True
                continue
            if t.startswith(";;#ASMEND"):
                inside = False
                continue
            if inside:
                has_copy |= "global_load_lds_dwordx4" in t
            elif t and not t.startswith(";") and re.search(r"\bm0\b", t):
                stray.append(t)
        if has_copy:
            checked += 1
            assert not stray, f"{name}: compiler-emitted M0 uses beside the inline copies: {stray[:3]}"
    assert checked > 0, "no kernel with the inline copy found"
