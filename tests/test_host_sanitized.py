"""The host core under AddressSanitizer + UBSan (CPU only).

Builds the node table, planner and C-ABI bookkeeping with g++ sanitizers
(kernel launchers stubbed) and runs the metadata and error-path suites
against that build in a subprocess with the sanitizer runtimes preloaded.
"""

import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _runtime(name):
    out = subprocess.run(["g++", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return out if os.path.isabs(out) and os.path.exists(out) else None


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_metadata_and_errors_under_asan_ubsan():
    sys.path.insert(0, ROOT)
    from paper_2508_17445_amd.build_host_sanitized import build
    lib = build()
    asan, ubsan = _runtime("libasan.so"), _runtime("libubsan.so")
    if not asan or not ubsan:
        pytest.skip("sanitizer runtimes not found")
    env = dict(os.environ)
    env.update(TREEPO_LIBRARY=lib, LD_PRELOAD=f"{asan}:{ubsan}",
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", TREEPO_NO_GPU_PROBE="1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        "tests/test_metadata.py", "tests/test_errors.py"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, tail
    assert "ERROR: AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, tail
