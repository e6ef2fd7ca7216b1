"""Segment-tree decode attention for TreePO rollouts on MI355X (gfx950).

The compute lives in ``libtreepo.so`` (HIP kernels behind the C-ABI of
``include/treepo.h``); ``treepo`` is its ctypes binding.
"""

from .treepo import (Context, TreePOError, load_library, bench_copy, bench_read, bench_stream,  # noqa: F401
                     bench_overlap,
                     branch_budget, BUDGET_EVEN, BUDGET_HIGH_PROB, BUDGET_LOW_PROB,
                     MODE_TREE, MODE_NAIVE, KERNEL_APPEND, KERNEL_PARTIAL, KERNEL_COMBINE, KERNEL_ADVANTAGE,
                     KERNEL_PREFILL,
                     ADV_MEAN, ADV_SIZE_WEIGHTED, NODE_FIELDS, BLOCK_TOKENS, LIB_PATH)
