"""CPU oracle of the vToken KV repack - TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.

A plain, slow, obviously correct host implementation of what one repack pass computes,
written from "vToken: Token-Level Virtualization for Reclaimable KV Caches" (arXiv
2608.13263). Only the test suite, the entry point's smoke check and the CPU-baseline leg of
the benchmark may import it. It shares no code with the HIP path and imports nothing from
it; the two meet only in the seeded inputs of paper_2608_13263_amd.workloads.

  repack.py      the vectorised numpy oracle: scan, admission, token table, copy, free list
  bruteforce.py  an independent per-token pure-Python version for tiny inputs
  invariants.py  convention-free checks of the paper's invariants I1, I2 and I4
  attention.py   dense vs paged decode attention over a cache (secondary check)

Parity status: every function here is pinned by tests that do not call back into it (brute
force on exhaustive tiny inputs, textbook reductions, the paper's printed block counts,
hand-derived worked examples and the invariant checkers); none is "parity unpinned".
"""
from .repack import (  # noqa: F401
    OracleResult,
    exclusive_live_rank,
    oracle_repack,
    plan_requests,
    slot_of_position,
    waste_ratio,
    block_live_counts,
    capacity_blocks,
    max_concurrency,
    kv_bytes_per_token,
)
from .bruteforce import brute_repack  # noqa: F401
from .invariants import check_invariants  # noqa: F401
