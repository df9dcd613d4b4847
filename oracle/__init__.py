"""fp64 CPU oracle for the strict-prefix linear-attention prefill.

TEST INFRASTRUCTURE ONLY.  Nothing in the product package imports this
package; only ``tests/``, ``__graft_entry__.smoke()`` and the cpu_baseline
leg of ``bench.py`` do.  It shares no code with the GPU path: the only module
both sides read is the seeded input generator, which holds none of the
method's arithmetic.

Contents
--------
* ``gdr_prefill``: the gated delta rule prefill, token by token in fp64,
  with checkpoints at multiples of the checkpoint interval (plain C in
  ``gdr_oracle.c``, loaded with ctypes).
* ``strict_prefix_boundary`` / ``nonstrict_lookup``: the paper's lookup
  rules by brute-force enumeration (``boundary.py``).
* ``paged_save`` / ``paged_restore``: the state pool as NumPy fancy
  indexing (``paging.py``).
* ``hybrid_boundary`` / ``hybrid_restore``: the joint attention-KV and
  recurrent-state boundary, by enumeration, and its restore as plain loops.
"""
from .gdr import gdr_prefill, gdr_prefill_seq, build_oracle, oracle_library_path  # noqa: F401
from .boundary import strict_prefix_boundary, nonstrict_lookup, hybrid_boundary  # noqa: F401
from .paging import paged_save, paged_restore, hybrid_restore  # noqa: F401
