"""Checks of the gfx950 code that the build produced (CPU only).

Scalar loads of bfloat16 weights read the aligned 32-bit word that holds a
value.  Where the compiler could prove an element index odd it once split such
an address into a base and an immediate offset that were each 2 mod 4, and the
load read the wrong word.  This test disassembles every kernel object of the
in-tree build and requires every scalar-load immediate offset to be a multiple
of 4.
"""
import glob
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BUILD = os.path.join(ROOT, "paper_1903_01814_amd", "_build")
LLVM = "/opt/rocm/llvm/bin"
TARGET = "hipv4-amdgcn-amd-amdhsa--gfx950"

SLOAD = re.compile(r"^\s*(s_load_\w+|s_buffer_load_\w+)\s+(.*)$")
IMM = re.compile(r"(?:offset:)?(0x[0-9a-fA-F]+|\d+)\s*$")


def _objects():
    return sorted(glob.glob(os.path.join(BUILD, "*.hip.o")))


def _disassemble(obj, tmp):
    fat = os.path.join(tmp, "fatbin")
    co = os.path.join(tmp, "code.o")
    subprocess.run([os.path.join(LLVM, "llvm-objcopy"), "--dump-section",
                    ".hip_fatbin=" + fat, obj, os.path.join(tmp, "host.o")],
                   check=True, capture_output=True)
    subprocess.run([os.path.join(LLVM, "clang-offload-bundler"), "--unbundle", "--type=o",
                    "--input=" + fat, "--targets=" + TARGET, "--output=" + co],
                   check=True, capture_output=True)
    r = subprocess.run([os.path.join(LLVM, "llvm-objdump"), "-d", "--mcpu=gfx950", co],
                       check=True, capture_output=True, text=True)
    return r.stdout


def misaligned_scalar_loads(text):
    """(instruction, operands) of scalar loads whose immediate offset is not
    a multiple of 4."""
    bad = []
    for line in text.splitlines():
        m = SLOAD.match(line.split("//")[0])
        if not m:
            continue
        ops = m.group(2).strip()
        im = IMM.search(ops)
        # operand list "sdst, sbase, offset": an immediate is the last field
        if im and ops.count(",") >= 2:
            v = int(im.group(1), 0)
            if v % 4:
                bad.append((m.group(1), ops))
    return bad


def test_parser_flags_half_word_offsets():
    text = ("\ts_load_dword s52, s[72:73], 0x2    // 0000: C0020D24 00000002\n"
            "\ts_load_dwordx8 s[12:19], s[0:1], 0x54\n"
            "\ts_load_dword s3, s[4:5], s6 offset:0x6\n"
            "\ts_load_dwordx2 s[8:9], s[0:1], 0x0\n")
    assert misaligned_scalar_loads(text) == [
        ("s_load_dword", "s52, s[72:73], 0x2"), ("s_load_dword", "s3, s[4:5], s6 offset:0x6")]


@pytest.mark.skipif(not _objects(), reason="no in-tree build (run __graft_entry__.build())")
@pytest.mark.skipif(not os.path.exists(os.path.join(LLVM, "llvm-objdump")),
                    reason="ROCm LLVM tools not installed")
@pytest.mark.parametrize("obj", _objects(), ids=os.path.basename)
def test_scalar_load_offsets_are_word_aligned(obj, tmp_path):
    text = _disassemble(obj, str(tmp_path))
    bad = misaligned_scalar_loads(text)
    assert not bad, "%d scalar loads with offsets not a multiple of 4, e.g. %s" % (
        len(bad), bad[:3])
