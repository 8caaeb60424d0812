"""Oracle row coalescing for computation deduplication (Sec. 4.2).

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper runs one forward pass per distinct token prefix instead of one per logical candidate:
a single explicit sequence carries a "potential size" n that stands for n identical candidates.
At the attention boundary this means: candidates whose block tables are identical (identical
token paths give identical tables once sealed steps are deduplicated) and whose query lengths are
equal are submitted once, as one row carrying a multiplicity.  Rows are numbered in order of first
appearance among the candidates.
"""
from __future__ import annotations

from typing import List, Sequence, Tuple


def coalesce(tables: Sequence[Sequence[int]], q_lens: Sequence[int]) -> Tuple[List[int], List[int], List[int]]:
    """Returns (row_of_candidate, first candidate of each row, multiplicity of each row)."""
    first: dict = {}
    row_of, rep, mult = [], [], []
    for c, (t, q) in enumerate(zip(tables, q_lens)):
        key = (int(q), tuple(int(b) for b in t))
        r = first.get(key)
        if r is None:
            r = len(rep)
            first[key] = r
            rep.append(c)
            mult.append(0)
        mult[r] += 1
        row_of.append(r)
    return row_of, rep, mult
