"""Builds the host core with AddressSanitizer + UBSan (CPU only, g++).

Produces ``_build/libtreepo_host_asan.so``: node table, planner and C-ABI
bookkeeping compiled for the host with sanitizers, kernel launchers replaced
by stubs.  ``tests/test_host_sanitized.py`` runs the metadata and error-path
suites against it in a subprocess with the sanitizer runtime preloaded.
"""

from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
OUT = os.path.join(HERE, "_build", "libtreepo_host_asan.so")


def build() -> str:
    os.makedirs(os.path.dirname(OUT), exist_ok=True)
    srcs = [os.path.join(HERE, "csrc", f) for f in ("tree_core.cpp", "treepo_api.cpp", "host_stub_launch.cpp")]
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fPIC", "-shared", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-D__HIP_PLATFORM_AMD__",
           f"-I{os.path.join(ROOT, 'include')}", f"-I{os.path.join(HERE, 'csrc')}", "-I/opt/rocm/include",
           *srcs, "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib", "-o", OUT]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(r.stdout + r.stderr)
    return OUT


if __name__ == "__main__":
    print(build())
