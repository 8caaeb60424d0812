"""Oracle: plain, slow, obviously-correct CPU reference for tree-shared paged attention.

TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the benchmark's CPU-baseline
leg may import this package.  The product path (the HIP library and its Python binding) never
imports, calls or links anything here, and this package imports nothing from the product.

Contents
  block_manager  prefix-tree KV block manager (dedup key, refcounts, lowest-free allocation, prune)
  attention      fp64 gather attention: each row's full KV by block table, no sharing
  coalesce       computation-deduplication row coalescing (identical candidates submitted once)
  kv_append      new tokens' K/V rows written to their pool slots (deduplicated blocks skipped)
  cd_sample      computation-deduplication branching: potential-many draws from one row, grouped
  search         speculative beam-search controller: early pruning and lazy verification

Pins: every function here is checked in tests/test_oracle.py against values that do not come from
this package (brute force in pure Python, closed forms, invariants, hand-worked fixtures under
tests/golden/).
"""
from .attention import attention, gather_kv
from .block_manager import BlockManager, BMError
from .coalesce import coalesce
from . import cd_sample
from . import search
from .kv_append import kv_append

__all__ = ["attention", "gather_kv", "BlockManager", "BMError", "coalesce", "kv_append", "cd_sample", "search"]
