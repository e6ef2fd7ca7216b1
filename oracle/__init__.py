"""fp64 CPU oracle for segment-tree decode attention.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import this
package: only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s
``cpu_baseline`` leg use it.  It shares no code with the HIP library.

What it computes follows TreePO (arXiv 2508.17445):

* ``metadata`` -- the segment tree itself: a root per query (depth 0),
  children forked from a path before each segment step, one segment of at
  most ``l`` tokens appended per node (Sec. 2.2 preliminaries and Alg. 1), and
  the per-leaf chain whose concatenated segments form the trajectory (the
  segment decomposition equation in Sec. 2.3).  The node->descendant-leaf sets
  are the nested subgroups G_j of Sec. 2.3 (Eq. groups).  Block reservation
  and id assignment are this library's documented rules.
* ``attention`` -- the plain definition: every leaf's query attends, with
  textbook softmax, over the concatenation of its chain's K/V rows.  Sharing
  a prefix changes where bytes come from, never the result (Sec. 2.1: shared
  prefixes are represented once).
* ``cascade`` -- the log-sum-exp algebra that lets per-node partial results be
  merged into the per-leaf result; it is pinned against ``attention``.
* ``advantage`` -- the TreePO advantage over the same descendant sets
  (Sec. 2.3, Eq. tree_ae; the size-weighted variant Eq. tree_ae_sgw).
* ``budget`` -- the branching budget over active paths (Sec. 2.2, Sec. 4.4).
* ``prefill`` -- causal attention of newly appended tokens over their chain
  (the shared prompt prefilled once for all rollouts of a query).
"""

from . import metadata, attention, cascade, advantage, prefill  # noqa: F401
