"""Oracle CD branching sampler: potential-many draws from one row's logits, grouped by token.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Computation deduplication (Sec. 4.2): a sequence with potential size n stands for n identical
candidates.  One decode step over it gives one row of logits; n tokens are then drawn from that one
distribution, each an independent trial, and equal tokens are grouped: each group becomes one
child whose potential is the group's size.  The distribution is the temperature softmax of the
logits (Sec. 2.1): p_j = exp(l_j / T) / sum_i exp(l_i / T).

A draw is the inverse CDF at a uniform u in [0, 1): the smallest token j whose cumulative
probability p_0 + ... + p_j exceeds u.  The uniforms are inputs, so a draw is a function of them.
Arithmetic in float64; tokens with probability 0 (logit -inf) are never drawn.
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

import numpy as np


def probabilities(logits: np.ndarray, temperature: float) -> np.ndarray:
    """Temperature softmax of one row, float64."""
    x = np.asarray(logits, dtype=np.float64) / float(temperature)
    e = np.exp(x - x.max())
    return e / e.sum()


def draw(logits: np.ndarray, temperature: float, uniforms: Sequence[float]) -> List[int]:
    """Inverse-CDF draws of one row, one per uniform."""
    p = probabilities(logits, temperature)
    cdf = np.cumsum(p)
    last = int(np.nonzero(p > 0)[0][-1])
    return [min(int(np.searchsorted(cdf, float(u), side="right")), last) for u in uniforms]


def group(tokens: Sequence[int]) -> Tuple[List[int], List[int]]:
    """Distinct tokens in ascending order and how often each was drawn."""
    vals, counts = np.unique(np.asarray(tokens, dtype=np.int64), return_counts=True)
    return [int(v) for v in vals], [int(c) for c in counts]


def cd_sample(logits: np.ndarray, temperature: float, potential: Sequence[int], uniforms: np.ndarray):
    """Rows [n_rows, vocab]; row r takes uniforms[off_r : off_r + potential[r]] (off = prefix sum).
    Returns per row (tokens ascending, counts, the draws in uniform order)."""
    out, off = [], 0
    for r, n in enumerate(potential):
        d = draw(logits[r], temperature, uniforms[off:off + n])
        toks, counts = group(d)
        out.append((toks, counts, d))
        off += n
    return out
