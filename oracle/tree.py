"""Oracle tree bookkeeping (test infrastructure only).

A verify step scores a token tree: row 0 is the root (the last committed
token), every other row is a draft token whose parent is an earlier row.
The paper's sparse branch structure (Appendix, "Tree Structure and Temporal
mismatch") -- B branches of k drafts each hanging off one branch point -- is
one such tree; a plain draft chain is another.
"""
from __future__ import annotations

import numpy as np


def validate(parents) -> None:
    par = [int(p) for p in parents]
    if not par or par[0] != -1:
        raise ValueError("row 0 must be the root (parent -1)")
    for i, p in enumerate(par[1:], start=1):
        if not (0 <= p < i):
            raise ValueError(f"parent of row {i} must be an earlier row, got {p}")


def depths(parents) -> np.ndarray:
    validate(parents)
    d = np.zeros(len(parents), dtype=np.int64)
    for i in range(1, len(parents)):
        d[i] = d[int(parents[i])] + 1
    return d


def root_path(parents, i: int) -> list[int]:
    """Rows from the root down to row i (inclusive), by ascending depth."""
    out = []
    while i >= 0:
        out.append(int(i))
        i = int(parents[i])
    return out[::-1]


def children(parents, i: int) -> list[int]:
    return [j for j in range(len(parents)) if int(parents[j]) == i]
