"""The library's branching budget (treepo_branch_budget) against the oracle:
bit-exact integers on random inputs (host only)."""

import numpy as np
import pytest

from oracle import budget as B
from tests.lib_helpers import ensure_lib


@pytest.mark.parametrize("seed", range(20))
def test_matches_oracle(seed):
    ensure_lib()
    from paper_2508_17445_amd import branch_budget
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 40))
    total = int(rng.integers(0, 300))
    s = rng.normal(-30, 15, size=n).astype(np.float32)
    for mode, name in ((0, "even"), (1, "high"), (2, "low")):
        for T in (0.5, 2.0, 5.0):
            got = branch_budget(s, total, mode, T)
            want = B.branch_budget([float(x) for x in s], total, name, float(np.float32(T)))
            assert got == want, (mode, T, got, want)


def test_errors():
    ensure_lib()
    from paper_2508_17445_amd import TreePOError, branch_budget
    for args in (([], 4, 0), ([0.0], -1, 0), ([0.0], 4, 3), ([float("nan")], 4, 1)):
        with pytest.raises(TreePOError):
            branch_budget(*args)
    with pytest.raises(TreePOError):
        branch_budget([0.0, 1.0], 4, 1, 0.0)
