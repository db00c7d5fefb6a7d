"""Exact enumeration of a randomized walk over its uniforms.

The oracle walk records every comparison it makes against a uniform: an
accept test ``u[c] < threshold`` or an inverse-CDF draw whose outcome
changes at ``u = C_v / W``.  Treating the uniforms as independent U[0,1)
variables, this module partitions the unit cube into boxes on which every
recorded decision is constant (splitting a box at the first breakpoint that
falls strictly inside it, and re-running the walk at the midpoint), and
returns the exact probability of every outcome as the sum of box volumes.

Used by the distribution tests; it holds no arithmetic of the method.
"""
from __future__ import annotations

from collections import defaultdict

import numpy as np


def _breakpoints(event) -> list[float]:
    kind = event[0]
    if kind == "accept":
        return [float(event[2])]
    if kind == "draw":
        C, W = event[2], event[3]
        if W <= 0:
            return []
        return [float(c) / W for c in C]
    raise ValueError(kind)


def enumerate_outcomes(run, n_uniforms: int, project, relevant=None):
    """run(u) -> (result, trace); project(result) -> hashable outcome.

    relevant(result, trace) -> number of leading trace events that can
    change the projected outcome (default: all).  It is only trusted once
    every earlier event is constant on the box, which the splitting order
    guarantees.  Returns {outcome: probability}.
    """
    out = defaultdict(float)
    stack = [(np.zeros(n_uniforms), np.ones(n_uniforms))]
    while stack:
        lo, hi = stack.pop()
        mid = 0.5 * (lo + hi)
        res, trace = run(mid)
        n_rel = len(trace) if relevant is None else relevant(res, trace)
        split = None
        for ev in trace[:n_rel]:
            idx = ev[1]
            inner = sorted({b for b in _breakpoints(ev) if lo[idx] < b < hi[idx]})
            if inner:
                split = (idx, inner)
                break
        if split is None:
            out[project(res)] += float(np.prod(hi - lo))
            continue
        idx, inner = split
        edges = [lo[idx]] + inner + [hi[idx]]
        for a, b in zip(edges[:-1], edges[1:]):
            if b > a:
                nlo, nhi = lo.copy(), hi.copy()
                nlo[idx], nhi[idx] = a, b
                stack.append((nlo, nhi))
    return dict(out)
