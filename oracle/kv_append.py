"""Oracle K/V append: write new tokens' K and V rows into the paged pool.

TEST INFRASTRUCTURE ONLY (see the package docstring).

A decode loop computes the K and V of each new token and stores them where the block manager put
the token: block b, position p, stored as the pool slot b * block_size + p.  A slot of -1 marks a
token of a block that was a deduplication hit; that block already holds the K/V of the same tokens
on the same prefix (computation deduplication, Sec. 4.2), so nothing is written for it.
"""
from __future__ import annotations

import numpy as np


def kv_append(k_pool: np.ndarray, v_pool: np.ndarray, dst, k_new: np.ndarray, v_new: np.ndarray) -> None:
    """In place.  Pools [num_blocks, hkv, block_size, d]; k_new, v_new [n_tok, hkv, d]; dst [n_tok]."""
    bs = k_pool.shape[2]
    for t, slot in enumerate(np.asarray(dst).reshape(-1)):
        slot = int(slot)
        if slot < 0:
            continue
        b, p = divmod(slot, bs)
        k_pool[b, :, p, :] = k_new[t]
        v_pool[b, :, p, :] = v_new[t]
