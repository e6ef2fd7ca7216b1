"""Machine-code invariants of the node-partial kernel (CPU: compiles only).

The kernel's load pipeline is counted by hand: tiles are global->LDS loads
waited for with explicit vmcnt barriers that allow the two newest tiles to
stay in flight.  That only holds if the compiler adds no vector-memory loads
or waits of its own and spills nothing to scratch (scratch traffic is vector
memory too); these tests read the gfx950 assembly built with the library's
flags and check exactly that.
"""

from __future__ import annotations

import re
import sys

import pytest

from tests.conftest import ROOT

sys.path.insert(0, f"{ROOT}/paper_2508_17445_amd")


@pytest.fixture(scope="module")
def partial_kernels(tmp_path_factory):
    import build
    asm = open(build.device_asm("kernels.hip", str(tmp_path_factory.mktemp("asm")))).read().split("\n")
    out = {}
    for i, line in enumerate(asm):
        m = re.match(r"^(_ZN6treepo\S*partial_kernelILi(\d+)\S*):", line)
        if m:
            end = next(j for j in range(i, len(asm)) if asm[j].startswith(".Lfunc_end"))
            body = [x.strip() for x in asm[i + 1:end]]
            out[int(m.group(2))] = [x for x in body if x and not x.startswith((";", "."))]
    return out, "\n".join(asm)


def test_both_head_dims_present(partial_kernels):
    kernels, _ = partial_kernels
    assert sorted(kernels) == [64, 128]


def test_only_global_to_lds_loads(partial_kernels):
    """Tiles, the stream block and the live tiles' lengths all arrive by
    global->LDS loads (16-byte tile chunks, non-temporal; 4-byte lengths)."""
    kernels, _ = partial_kernels
    for d, body in kernels.items():
        loads = [x for x in body if re.match(r"^(global_load|buffer_load|flat_load|scratch_|global_atomic)", x)
                 and not re.match(r"^global_load_lds_dword(x4)?\s", x)]
        assert not loads, (d, loads[:5])
        assert any(x.startswith("global_load_lds_dwordx4") and x.endswith(" nt") for x in body), d


def test_no_scratch(partial_kernels):
    _, meta = partial_kernels
    sizes = re.findall(r"\.private_segment_fixed_size:\s+(\d+)\n(?:.*\n){0,40}?\s+\.symbol:\s+\S*partial_kernel", meta)
    assert len(sizes) == 2 and all(int(s) == 0 for s in sizes), sizes


def test_every_vector_memory_wait_is_a_pipeline_barrier(partial_kernels):
    kernels, _ = partial_kernels
    for d, body in kernels.items():
        for i, x in enumerate(body):
            if x.startswith("s_waitcnt") and "vmcnt" in x:
                assert re.match(r"^s_waitcnt vmcnt\(\d+\) lgkmcnt\(0\)$", x), (d, x)
                assert body[i + 1] == "s_barrier", (d, body[i:i + 2])


@pytest.fixture(scope="module")
def prefill_kernels(tmp_path_factory):
    import build
    asm = open(build.device_asm("kernels.hip", str(tmp_path_factory.mktemp("asm_pf")))).read()
    lines = asm.split("\n")
    out = {}
    for i, line in enumerate(lines):
        m = re.match(r"^(_ZN6treepo\S*prefill_kernelILi(\d+)\S*):", line)
        if m:
            end = next(j for j in range(i, len(lines)) if lines[j].startswith(".Lfunc_end"))
            body = [x.strip() for x in lines[i + 1:end]]
            out[int(m.group(2))] = [x for x in body if x and not x.startswith((";", "."))]
    return out, asm


def test_prefill_pipeline_waits(prefill_kernels):
    """The prefill kernel's query rows are plain loads waited for before the
    first tile is issued; after that every vector-memory wait is a tile
    barrier, so the three tiles in flight are never drained by the compiler."""
    kernels, asm = prefill_kernels
    assert sorted(kernels) == [64, 128]
    for d, body in kernels.items():
        first_dma = next(i for i, x in enumerate(body) if x.startswith("global_load_lds_dwordx4"))
        plain = [i for i, x in enumerate(body) if re.match(r"^(global_load|buffer_load|flat_load|scratch_)", x)
                 and not x.startswith("global_load_lds")]
        assert plain and max(plain) < first_dma, d
        for i, x in enumerate(body[first_dma:]):
            if x.startswith("s_waitcnt") and "vmcnt" in x:
                assert re.match(r"^s_waitcnt vmcnt\(\d+\) lgkmcnt\(0\)$", x), (d, x)
                assert body[first_dma + i + 1] == "s_barrier", (d, body[first_dma + i:first_dma + i + 2])
    sizes = re.findall(r"\.private_segment_fixed_size:\s+(\d+)\n(?:.*\n){0,40}?\s+\.symbol:\s+\S*prefill_kernel", asm)
    assert len(sizes) == 2 and all(int(s) == 0 for s in sizes), sizes
