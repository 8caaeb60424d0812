"""Oracle attention: fp64 gather attention over a paged KV cache, with no sharing.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Definition (the textbook scaled dot-product attention the paper's serving substrate runs,
Sec. 2.1; verification is a prefill-only pass over the new step's tokens, Sec. 3.2.2).  For a row
with block table T, q_len L and kv_len N = sum of block_len over T:

  K, V      = concatenation over T, in order, of the first block_len[b] slots of block b
  kvh(h)    = floor(h / G),  G = Hq / Hkv  (consecutive query heads share a KV head)
  s_j       = <q[i, h], K[j, kvh]> / sqrt(d)      for j in [0, N - L + i]  (bottom-right causal;
                                                   decode is L = 1 and sees all N keys)
  o[i, h]   = sum_j softmax(s)_j V[j, kvh]
  lse[i, h] = log sum_j exp(s_j)                  (natural log)

Arithmetic is float64 on the exact input values (the bf16 inputs widen exactly), with the row
maximum subtracted before exponentiation.  Each row re-gathers its whole path: shared blocks are
read once per row that references them, which is exactly the work the method avoids.
"""
from __future__ import annotations

import math
from typing import Sequence, Tuple

import numpy as np


def gather_kv(pool: np.ndarray, table: Sequence[int], block_len: Sequence[int]) -> np.ndarray:
    """[num_blocks, Hkv, bs, d] pool -> [Hkv, N, d] float64 keys (or values) of one path."""
    parts = [pool[b, :, :block_len[b], :] for b in table]
    return np.concatenate(parts, axis=1).astype(np.float64)


def attention(q: np.ndarray, k_pool: np.ndarray, v_pool: np.ndarray,
              tables: Sequence[Sequence[int]], block_len: Sequence[int], q_lens: Sequence[int],
              rows: Sequence[int] = None) -> Tuple[np.ndarray, np.ndarray]:
    """q: [n_qtok, Hq, d] (query tokens of all rows, row-major by q_lens); pools [nb, Hkv, bs, d].

    Returns (o [n_qtok, Hq, d], lse [n_qtok, Hq]) in float64.  `rows`, if given, restricts the
    computation to those rows (other entries are left NaN) -- used to time a bounded sample.
    """
    n_qtok, hq, d = q.shape
    hkv = k_pool.shape[1]
    if hq % hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    g = hq // hkv
    scale = 1.0 / math.sqrt(d)
    qoff = np.concatenate([[0], np.cumsum(q_lens)]).astype(np.int64)
    if qoff[-1] != n_qtok:
        raise ValueError("q_lens do not add up to the number of query tokens")
    o = np.full((n_qtok, hq, d), np.nan)
    lse = np.full((n_qtok, hq), np.nan)
    for r in (range(len(tables)) if rows is None else rows):
        L = int(q_lens[r])
        K = gather_kv(k_pool, tables[r], block_len)
        V = gather_kv(v_pool, tables[r], block_len)
        N = K.shape[1]
        if not 1 <= L <= N:
            raise ValueError(f"row {r}: need 1 <= q_len <= kv_len (q_len {L}, kv_len {N})")
        qr = q[qoff[r]:qoff[r] + L].astype(np.float64)                 # [L, Hq, d]
        # token i sees keys 0 .. N - L + i
        visible = np.arange(N)[None, :] <= (N - L + np.arange(L))[:, None]    # [L, N]
        for kvh in range(hkv):
            Q = qr[:, kvh * g:(kvh + 1) * g, :]                          # [L, G, d]
            S = (Q.reshape(L * g, d) @ K[kvh].T).reshape(L, g, N) * scale  # [L, G, N]
            S = np.where(visible[:, None, :], S, -np.inf)
            m = S.max(axis=2, keepdims=True)
            P = np.exp(S - m)
            l = P.sum(axis=2, keepdims=True)
            PV = (P.reshape(L * g, N) @ V[kvh]).reshape(L, g, d)
            o[qoff[r]:qoff[r] + L, kvh * g:(kvh + 1) * g, :] = PV / l
            lse[qoff[r]:qoff[r] + L, kvh * g:(kvh + 1) * g] = (m + np.log(l))[..., 0]
    return o, lse
