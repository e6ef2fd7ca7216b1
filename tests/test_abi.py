"""The shared library loads and exports every symbol the public headers declare."""

import os
import re

from tests.lib_helpers import ensure_lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    names = set()
    for h in ("treepo.h", "treepo_bench.h"):
        with open(os.path.join(ROOT, "include", h)) as f:
            text = f.read()
        names |= set(re.findall(r"^\s*(?:int32_t|const char\*|size_t)\s+(treepo_\w+)\s*\(", text, re.M))
    return names


def test_headers_declare_the_boundary():
    names = _declared()
    for must in ("treepo_kv_append", "treepo_fork", "treepo_tree_decode", "treepo_paged_decode_naive",
                 "treepo_new_root", "treepo_export_chains", "treepo_export_nodes"):
        assert must in names


def test_library_exports_every_declared_symbol():
    lib = ensure_lib()
    missing = [n for n in sorted(_declared()) if not hasattr(lib, n)]
    assert not missing, missing


def test_strerror_covers_every_code():
    lib = ensure_lib()
    for code in range(-8, 1):
        assert lib.treepo_strerror(code).decode() != "unknown status"
