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


def worker_threads() -> int:
    """Threads for host-side checking: this process's CPUs, at most 16 (one GPU's share of a box)."""
    import os
    return max(1, min(16, len(os.sched_getaffinity(0))))


def oracle_check(q_bits, k_f32, v_f32, tables, block_len, q_lens, o, lse, rows=None, threads=None):
    """Compare device results with the oracle, row by row.

    The oracle runs on sub-batches of rows in parallel threads (BLAS single-threaded inside each):
    rows are independent in the definition, so a sub-batch computes exactly what the whole batch
    would for those rows.  q_bits: [n_qtok, hq, d] bf16 bits; k_f32 / v_f32: the pools widened to
    float32; o, lse: the device results as float32 arrays.  Returns a dict with the max and mean
    absolute error of o, the max absolute error of lse, the number of tokens compared and whether
    every compared output is finite."""
    from concurrent.futures import ThreadPoolExecutor
    from threadpoolctl import threadpool_limits
    import oracle
    qoff = np.concatenate([[0], np.cumsum(q_lens)]).astype(np.int64)
    rows = list(range(len(tables))) if rows is None else list(rows)
    threads = threads or worker_threads()
    # cost-balanced sub-batches: rows by decreasing q_len * kv_len, dealt round-robin
    cost = {r: int(q_lens[r]) * sum(int(block_len[b]) for b in tables[r]) for r in rows}
    order = sorted(rows, key=lambda r: -cost[r])
    n_sub = max(1, min(len(rows), 8 * threads))
    subs = [order[i::n_sub] for i in range(n_sub)]

    def run(sub):
        idx = np.concatenate([np.arange(qoff[r], qoff[r + 1]) for r in sub])
        qs = W.bf16_bits_to_f32(q_bits[idx]).astype(np.float64)
        o_ref, l_ref = oracle.attention(qs, k_f32, v_f32, [tables[r] for r in sub], block_len,
                                        [int(q_lens[r]) for r in sub])
        og, lg = o[idx], lse[idx]
        err = np.abs(og - o_ref)
        lerr = np.abs(lg - l_ref)
        return (float(err.max()), float(err.sum()), int(err.size), float(lerr.max()),
                bool(np.isfinite(og).all() and np.isfinite(lg).all()), len(idx))

    with threadpool_limits(1):
        with ThreadPoolExecutor(threads) as ex:
            res = list(ex.map(run, [s for s in subs if s]))
    return {"max": max(r[0] for r in res), "mean": sum(r[1] for r in res) / sum(r[2] for r in res),
            "lse_max": max(r[3] for r in res), "finite": all(r[4] for r in res),
            "tokens": sum(r[5] for r in res)}
