"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU
only): the fp64 oracle (oracle/hexoracle.c, every 2-D and 3-D entry point)
and the library's host geometry and generic launch plans (csrc/hexgeom.h,
csrc/generic_plan.h), each built with gcc/g++ -fsanitize=address,undefined
and driven over many kernel sizes, strides and ragged shapes.  A finding
aborts the driver and fails the test."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
NATIVE = os.path.join(ROOT, "tests", "native")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
       "-g", "-O1"]


def _run(cmd_build, exe):
    r = subprocess.run(cmd_build, capture_output=True, text=True)
    if r.returncode != 0:
        if "cannot find" in r.stderr and "asan" in r.stderr:
            pytest.skip("sanitizer runtime not installed")
        raise AssertionError(r.stderr)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1", OMP_NUM_THREADS="2")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, r.stdout + r.stderr
    return r.stdout


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "san_oracle")
    out = _run(["gcc", "-std=c99", "-fopenmp"] + SAN +
               [os.path.join(ROOT, "oracle", "hexoracle.c"),
                os.path.join(NATIVE, "sanitize_oracle.c"), "-o", exe], exe)
    assert "ok" in out


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_host_geometry_under_sanitizers(tmp_path):
    exe = str(tmp_path / "san_geom")
    out = _run(["g++", "-std=c++17"] + SAN +
               ["-I", os.path.join(ROOT, "paper_1903_01814_amd", "csrc"),
                os.path.join(NATIVE, "sanitize_geom.cpp"), "-o", exe], exe)
    assert "ok" in out
