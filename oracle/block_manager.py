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

Growing a path token by token (a decode loop) and completing a step:

* append(seq, tokens) grows the sequence in place.  Its open (unsealed) step is private to it -- no
  sequence can be extended from an unsealed one -- so the tokens fill the open step's last block and
  then take the lowest free ids, one block at a time.  A sealed sequence starts a new open step in a
  fresh block (step-aligned, as for extensions).  Open blocks are never indexed.
* seal(seq) completes the open step: its blocks, in path order, are looked up with the dedup key
  above (the predecessor being the block the path now holds there).  A hit replaces the sequence's
  own block with the live sealed block of the same key (whose refcount rises; the own block, held
  by this sequence only, is freed); a miss indexes the block.  As in an extension, once a block
  misses every later one misses (a block that was just indexed precedes nothing in the index).
* fork(seq, tokens) branches a sequence where its candidates' next tokens differ (the on-demand
  branching of Sec. 4.2): the open step, if any, is sealed there -- the point of divergence becomes a
  step boundary, so the children share every block before it -- and each token starts one child, a
  new sequence whose open step holds that token.  The children take the lowest free sequence ids in
  token order.  Nothing changes unless every child gets its block and sequence slot.
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
        self.seqs: Dict[int, dict] = {}                          # seq -> {table, sealed, open}
        # "open": tokens of the open (unsealed) step, which fill the last ceil(len / block_size)
        # blocks of the table (empty for a sealed sequence)

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
        self.seqs[seq] = {"table": table, "sealed": bool(seal), "open": [] if seal else list(toks)}
        return seq, new_ids, hits

    def append(self, seq: int, tokens) -> List[int]:
        """Grow `seq` in place by `tokens`; returns each token's pool slot, block * block_size + slot."""
        toks = [int(t) for t in np.asarray(tokens).reshape(-1)]
        if seq not in self.seqs:
            raise BMError(ENOSEQ, f"unknown sequence {seq}")
        sq = self.seqs[seq]
        bs = self.block_size
        open_toks = [] if sq["sealed"] else sq["open"]
        room = (-len(open_toks)) % bs            # free slots in the open step's last block
        need = -(-max(0, len(toks) - room) // bs)
        if need > len(self.free_blocks):
            raise BMError(ENOMEM, f"pool exhausted: need {need} blocks, {len(self.free_blocks)} free")
        if sq["sealed"]:
            sq["sealed"] = False
            sq["open"] = open_toks = []
        dst = []
        for t in toks:
            if len(open_toks) % bs == 0:          # the open step's last block is full (or there is none)
                b = heapq.heappop(self.free_blocks)
                self.refcount[b] = 1
                sq["table"].append(b)
            b = sq["table"][-1]
            dst.append(b * bs + self.block_len[b])
            self.block_len[b] += 1
            open_toks.append(t)
        return dst

    def fork(self, seq: int, tokens) -> List[int]:
        """Branch `seq`: seal its open step, then one open child per token.  Returns the children."""
        toks = [int(t) for t in np.asarray(tokens).reshape(-1)]
        if seq not in self.seqs:
            raise BMError(ENOSEQ, f"unknown sequence {seq}")
        if len(toks) > len(self.free_blocks) or len(toks) > len(self.free_seqs):
            raise BMError(ENOMEM, f"fork into {len(toks)} children: {len(self.free_blocks)} blocks, "
                                  f"{len(self.free_seqs)} sequence slots free")
        if not self.seqs[seq]["sealed"]:
            self.seal(seq)
        return [self.extend(seq, [t], False)[0] for t in toks]

    def seal(self, seq: int) -> List[Tuple[int, int]]:
        """Complete the open step of `seq`; returns the (own block, live sealed block) replacements."""
        if seq not in self.seqs:
            raise BMError(ENOSEQ, f"unknown sequence {seq}")
        sq = self.seqs[seq]
        if sq["sealed"]:
            raise BMError(EINVAL, f"sequence {seq} is already sealed")
        bs = self.block_size
        table, open_toks = sq["table"], sq["open"]
        n_open = -(-len(open_toks) // bs)
        first = len(table) - n_open
        replaced = []
        for j in range(n_open):
            i = first + j
            pred = table[i - 1] if i > 0 else -1
            key = (pred, tuple(open_toks[j * bs:(j + 1) * bs]))
            own = table[i]
            hit = self.index.get(key)
            if hit is not None:
                table[i] = hit
                self.refcount[hit] += 1
                self.refcount[own] = 0
                self.block_len[own] = 0
                heapq.heappush(self.free_blocks, own)
                replaced.append((own, hit))
            else:
                self.key[own] = key
                self.index[key] = own
        sq["sealed"] = True
        sq["open"] = []
        return replaced

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
            "seqs": {s: (tuple(v["table"]), int(v["sealed"]), -(-len(v["open"]) // self.block_size))
                     for s, v in sorted(self.seqs.items())},
        }
