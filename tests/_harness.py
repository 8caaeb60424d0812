"""Test plumbing: realise a seeded workload on a block manager and lay out the attention inputs.

Each side runs the workload's script on its own block manager: the oracle side on
oracle.BlockManager with oracle.coalesce, the library side on the C block manager with
tkv_bm_coalesce.  Only the seeded values from `workloads` are shared.
"""
from dataclasses import dataclass
from typing import List

import numpy as np

import workloads as W


@dataclass
class Batch:
    """One launch after coalescing: rows in first-appearance order."""
    launch: W.Launch
    index: int
    tables: List[List[int]]
    q_lens: List[int]
    mult: List[int]
    block_len: np.ndarray
    decode: bool

    @property
    def n_qtok(self):
        return int(sum(self.q_lens))

    def arrays(self):
        q_indptr = np.concatenate([[0], np.cumsum(self.q_lens)]).astype(np.int32)
        kv_indptr = np.concatenate([[0], np.cumsum([len(t) for t in self.tables])]).astype(np.int32)
        kv_blocks = (np.concatenate([np.asarray(t, dtype=np.int32) for t in self.tables])
                     if self.tables else np.zeros(0, dtype=np.int32))
        return q_indptr, kv_indptr, kv_blocks


def realize(wl: W.Workload, bm, coalesce) -> List[Batch]:
    """Run the script on `bm`; `coalesce(bm, seqs, q_lens) -> (row_of, first, mult)`."""
    out = []

    def on_launch(i, launch, cands):
        seqs = [s for s, _ in cands]
        qls = [q for _, q in cands]
        _, first, mult = coalesce(bm, seqs, qls)
        tables = [[int(b) for b in bm.table(seqs[c])] for c in first]
        if hasattr(bm, "block_len") and callable(bm.block_len):
            bl = np.asarray(bm.block_len(), dtype=np.int32)
        else:
            bl = np.asarray(bm.block_len, dtype=np.int32)
        out.append(Batch(launch, i, tables, [qls[c] for c in first], [int(m) for m in mult], bl.copy(), launch.decode))

    W.drive(wl, bm, on_launch=on_launch)
    return out


def realize_oracle(wl: W.Workload):
    import oracle
    bm = oracle.BlockManager(wl.num_blocks, wl.shape.block_size, wl.max_seqs)
    return realize(wl, bm, lambda b, s, q: oracle.coalesce([b.table(x) for x in s], q))


def realize_native(wl: W.Workload):
    import paper_2609_39334_amd as tkv
    bm = tkv.BlockManager(wl.num_blocks, wl.shape.block_size, wl.max_seqs)
    return realize(wl, bm, lambda b, s, q: b.coalesce(s, q))
