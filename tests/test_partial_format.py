"""The block floating-point format of compact plans' partial rows
(`csrc/partial_format.h`, compiled for the host): its bit layout on
hand-worked groups and its error bound -- each decoded value within 2^-13 of
its group's largest magnitude -- on two million random groups across the
fp32 exponent range.  The decode kernels use the same header; the GPU parity
tests check the merged outputs against the oracle."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _hipcc():
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    return None


@pytest.mark.skipif(_hipcc() is None, reason="needs hipcc")
def test_partial_row_format(tmp_path):
    exe = str(tmp_path / "partial_format_check")
    build = subprocess.run([_hipcc(), "-x", "hip", "--offload-host-only", "-O2", "-std=c++17",
                            "-I", os.path.join(ROOT, "paper_2508_17445_amd", "csrc"),
                            os.path.join(ROOT, "tests", "native", "partial_format_check.cpp"), "-o", exe],
                           capture_output=True, text=True, timeout=300)
    assert build.returncode == 0, build.stderr[-3000:]
    run = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    assert run.returncode == 0 and run.stdout.startswith("ok "), run.stdout + run.stderr
    assert float(run.stdout.split()[1]) <= 2.0 ** -13
