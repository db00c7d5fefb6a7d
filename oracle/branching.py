"""Oracle of the branch-point candidates (test infrastructure only).

Section "Branch Resampling": at an unconfident draft token x_b the draft
side spawns parallel branches whose first tokens are resampled from the
draft's distribution q at that position, B = max(1, floor(k_max (1 -
q(x_b)))) of them (k_max about 6, Section "Experiments", "Resource
Consumption").  Verification (Algorithm 1) subtracts from p the
distribution each candidate was drawn from, so each candidate carries its
own q row (reading R1):

  "topk" -- the B largest entries of q (ties: lowest index first); the
            choice is deterministic, so each candidate's row is one-hot;
  "iid"  -- B independent inverse-CDF draws from q with u[0..B-1]; every
            candidate carries q itself;
  "wor"  -- draws without replacement: candidate i is drawn from q with the
            earlier candidates zeroed, and carries that remainder
            normalised, float32(r_v / Z) with Z the float64 sum of r.

B is computed in float64 from the float32 q(x_b) and never exceeds the
number of tokens with q > 0.  Draws follow sampling.draw (float64 running
sums in vocabulary order, first index whose sum exceeds u * W).
"""
from __future__ import annotations

import math

import numpy as np

from .sampling import draw

MODES = ("topk", "iid", "wor")


def branch_count(q_xb: float, k_max: int, n_positive: int | None = None) -> int:
    b = max(1, int(math.floor(float(k_max) * (1.0 - float(np.float32(q_xb))))))
    return min(b, n_positive) if n_positive is not None else b


def candidates(q_row, x_b: int, k_max: int, mode: str, u, trace: list | None = None):
    """(tokens [B] int32, rows [B][V] float32).  With `trace`, each draw is
    recorded as sampling.draw records it (uniform index i for candidate i)."""
    q = np.asarray(q_row, dtype=np.float32)
    V = len(q)
    nnz = int(np.count_nonzero(q > 0))
    B = branch_count(q[x_b], k_max, nnz)
    rows = np.zeros((B, V), dtype=np.float32)
    toks = np.zeros(B, dtype=np.int32)
    if mode == "topk":
        order = np.argsort(-q.astype(np.float64), kind="stable")
        for i in range(B):
            toks[i] = order[i]
            rows[i, toks[i]] = 1.0
    elif mode == "iid":
        for i in range(B):
            toks[i] = draw(q.astype(np.float64), float(u[i]), trace, i)
            rows[i] = q
    elif mode == "wor":
        rem = q.astype(np.float64).copy()
        for i in range(B):
            Z = float(np.sum(rem))
            rows[i] = (rem / Z).astype(np.float32)
            toks[i] = draw(rem, float(u[i]), trace, i)
            rem[toks[i]] = 0.0
    else:
        raise ValueError(mode)
    return toks, rows
