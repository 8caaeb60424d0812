"""Oracle block manager: the prefix tree of reasoning-step blocks over one paged KV pool.

TEST INFRASTRUCTURE ONLY (see the package docstring).

What the paper fixes: candidates of one request share the KV cache of their common prefix
(prefix KV caching and sharing with paged attention, Sec. 5.1 setup); identical candidates are
one explicit sequence (computation deduplication, Sec. 4.2); pruning ends a path and releases what
only it used (early pruning, Sec. 4.1; lower KV usage, Sec. 5.7).  The paper gives no block-level
rules, so the following reading is used and is exact (no hashing decides anything):

* Step-aligned blocks: each extension starts a fresh block; n tokens take ceil(n/16) blocks and the
  last one may be partial (block_len < 16).
* Dedup key of a chunk = (id of the preceding block in the path, or -1 at a root; the chunk's exact
  tokens).  A chunk of a *sealed* extension reuses the live sealed block with the same key (a hit);
  otherwise it takes the lowest free block id (a miss).  Chunks of unsealed (in-progress) extensions
  never hit and are never indexed.
* refcount(b) = number of live sequences whose table contains b.  A block whose refcount reaches 0
  is freed at once and leaves the index (no cached-but-free pool).
* New sequence id = lowest free id.  Extending an unsealed sequence is an error; so is a root with no
  tokens.  Errors leave the state unchanged.
"""
from __future__ import annotations

import heapq
from typing import Dict, List, Optional, Tuple

import numpy as np

EINVAL, ENOMEM, ENOSEQ = -1, -2, -3


class BMError(Exception):
    def __init__(self, code: int, msg: str):
        super().__init__(msg)
        self.code = code


class BlockManager:
    def __init__(self, num_blocks: int, block_size: int = 16, max_seqs: int = 1024):
        if num_blocks < 1 or block_size < 1 or max_seqs < 1:
            raise BMError(EINVAL, "bad sizes")
        self.num_blocks = num_blocks
        self.block_size = block_size
        self.max_seqs = max_seqs
        self.refcount = [0] * num_blocks
        self.block_len = [0] * num_blocks
        self.key: List[Optional[tuple]] = [None] * num_blocks   # set iff the block is indexed
        self.index: Dict[tuple, int] = {}
        self.free_blocks = list(range(num_blocks))              # a heap: lowest id first
        self.free_seqs = list(range(max_seqs))
        self.seqs: Dict[int, dict] = {}                          # seq -> {table, sealed}

    # ------------------------------------------------------------------ operations
    def extend(self, parent: int, tokens, seal: bool) -> Tuple[int, List[int], List[int]]:
        """New sequence = parent's path + tokens.  Returns (seq, new block ids, hit flags)."""
        toks = [int(t) for t in np.asarray(tokens).reshape(-1)]
        if parent == -1:
            if not toks:
                raise BMError(EINVAL, "a root needs at least one token")
            table: List[int] = []
        else:
            if parent not in self.seqs:
                raise BMError(ENOSEQ, f"unknown parent sequence {parent}")
            if not self.seqs[parent]["sealed"]:
                raise BMError(EINVAL, "cannot extend an unsealed (in-progress) sequence")
            table = list(self.seqs[parent]["table"])
        if not self.free_seqs:
            raise BMError(ENOMEM, "no free sequence slot")
        bs = self.block_size
        chunks = [tuple(toks[i:i + bs]) for i in range(0, len(toks), bs)]
        # Resolve hits first (a miss can never be followed by a hit: a freshly allocated block is
        # nobody's predecessor yet), so the allocation need is known before anything changes.
        pred = table[-1] if table else -1
        plan = []
        for c in chunks:
            hit = self.index.get((pred, c)) if seal else None
            if hit is None:
                break
            plan.append(hit)
            pred = hit
        n_miss = len(chunks) - len(plan)
        if n_miss > len(self.free_blocks):
            raise BMError(ENOMEM, f"pool exhausted: need {n_miss} blocks, {len(self.free_blocks)} free")
        # Commit.
        seq = heapq.heappop(self.free_seqs)
        for b in table:
            self.refcount[b] += 1
        new_ids, hits = [], []
        pred = table[-1] if table else -1
        for i, c in enumerate(chunks):
            if i < len(plan):
                b = plan[i]
                hits.append(1)
            else:
                b = heapq.heappop(self.free_blocks)
                self.block_len[b] = len(c)
                if seal:
                    self.key[b] = (pred, c)
                    self.index[(pred, c)] = b
                hits.append(0)
            self.refcount[b] += 1
            table.append(b)
            new_ids.append(b)
            pred = b
        self.seqs[seq] = {"table": table, "sealed": bool(seal)}
        return seq, new_ids, hits

    def prune(self, seq: int) -> List[int]:
        """Release a sequence; returns the block ids freed, in table order."""
        if seq not in self.seqs:
            raise BMError(ENOSEQ, f"unknown sequence {seq}")
        freed = []
        for b in self.seqs[seq]["table"]:
            self.refcount[b] -= 1
            if self.refcount[b] == 0:
                if self.key[b] is not None:
                    del self.index[self.key[b]]
                    self.key[b] = None
                self.block_len[b] = 0
                heapq.heappush(self.free_blocks, b)
                freed.append(b)
        del self.seqs[seq]
        heapq.heappush(self.free_seqs, seq)
        return freed

    # ------------------------------------------------------------------ queries
    def table(self, seq: int) -> List[int]:
        if seq not in self.seqs:
            raise BMError(ENOSEQ, f"unknown sequence {seq}")
        return list(self.seqs[seq]["table"])

    def kv_len(self, seq: int) -> int:
        return sum(self.block_len[b] for b in self.table(seq))

    def snapshot(self) -> dict:
        """Complete state for bit-exact comparison."""
        return {
            "refcount": np.array(self.refcount, dtype=np.int32),
            "block_len": np.array(self.block_len, dtype=np.int32),
            "indexed": np.array([k is not None for k in self.key], dtype=np.int32),
            "seqs": {s: (tuple(v["table"]), int(v["sealed"])) for s, v in sorted(self.seqs.items())},
        }
