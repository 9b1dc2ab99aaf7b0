"""Constraints on the generated gfx950 code that the sources rely on (CPU).

The inline-assembly global-to-LDS copy (dma16_opaque in csrc/common.h) sets
M0, a register the compiler reserves and does not take as clobbered.  Each
copy statement saves M0 in a scratch SGPR and restores it right after the
copy, so a value the compiler keeps in M0 survives it.  This test
cross-compiles every library source to assembly and checks, in every kernel
that contains the copy, that each statement restores M0 from the register it
saved it in, and that the compiler emits no M0 use of its own there either
(a second guard: none is needed today).
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


def _asm_blocks(body):
    """(inline-assembly blocks as lists of instructions, compiler lines outside them)."""
    blocks, outside, cur = [], [], None
    for line in body.splitlines():
        t = line.strip()
        if t.startswith(";;#ASMSTART"):
            cur = []
            continue
        if t.startswith(";;#ASMEND"):
            blocks.append(cur)
            cur = None
            continue
        if cur is not None:
            if t and not t.startswith(";"):
                cur.append(t)
        elif t and not t.startswith(";"):
            outside.append(t)
    return blocks, outside


_CHECKED = {}


@pytest.mark.parametrize("src", build.SOURCES)
def test_opaque_copies_keep_m0(src):
    asm = _device_asm(src)
    checked = 0
    for name, body in _kernels(asm):
        blocks, outside = _asm_blocks(body)
        copies = [b for b in blocks if any("global_load_lds_dwordx4" in t for t in b)]
        if not copies:
            continue
        checked += 1
        for b in copies:
            save = re.fullmatch(r"s_mov_b32\s+(s\d+),\s*m0", b[0])
            assert save, f"{name}: copy statement does not start by saving M0: {b}"
            reg = save.group(1)
            assert re.fullmatch(rf"s_mov_b32\s+m0,\s*{reg}", b[-1]), f"{name}: M0 not restored from {reg}: {b}"
            assert all(reg not in t for t in b[1:-1]), f"{name}: the saved register is reused inside: {b}"
        stray = [t for t in outside if re.search(r"\bm0\b", t)]
        assert not stray, f"{name}: compiler-emitted M0 uses beside the inline copies: {stray[:3]}"
    _CHECKED[src] = checked


def test_some_kernel_uses_the_opaque_copy():
    missing = [s for s in build.SOURCES if s not in _CHECKED]
    for src in missing:
        test_opaque_copies_keep_m0(src)
    assert sum(_CHECKED.values()) > 0, "no kernel with the inline copy found"
