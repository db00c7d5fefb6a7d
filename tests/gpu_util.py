"""Helpers for the GPU parity tests (no arithmetic of the method here)."""
from __future__ import annotations

import math
import sys

import numpy as np


def say(*a) -> None:
    """Progress line naming the case, flushed before a GPU step."""
    print(*a, flush=True)
    sys.stdout.flush()


def decision_margin(trace, u) -> float:
    """Smallest distance between a uniform and a decision threshold on the
    oracle's path (relative to the CDF total for draws)."""
    m = math.inf
    for ev in trace:
        if ev[0] == "accept":
            thr = ev[2]
            if np.isfinite(thr):
                m = min(m, abs(float(u[ev[1]]) - thr))
        else:
            C, W = ev[2], ev[3]
            if W > 0:
                t = float(u[ev[1]]) * W
                m = min(m, float(np.min(np.abs(C - t))) / W)
    return m


def row_relerr(a: np.ndarray, b: np.ndarray) -> float:
    """max over rows of max_v |a - b| / max_v |b| (per-row normwise)."""
    a = np.asarray(a, dtype=np.float64).reshape(a.shape[0], -1)
    b = np.asarray(b, dtype=np.float64).reshape(b.shape[0], -1)
    num = np.max(np.abs(a - b), axis=1)
    den = np.maximum(np.max(np.abs(b), axis=1), 1e-30)
    return float(np.max(num / den))
