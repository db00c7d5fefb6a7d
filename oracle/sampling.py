"""Oracle accept / select / resample (test infrastructure only).

What it follows in the paper:

* Preliminaries, "Speculative Decoding": a draft token x drawn from q is
  accepted with probability min(1, p(x)/q(x)); on rejection the later drafts
  are dropped and a token is drawn from norm(max(0, p - q)); if every draft
  is accepted one more token is drawn from the target distribution of the
  last position.
* Appendix "Branch Speculative Sampling", Algorithm 1: at a branch point the
  candidates x^1..x^B (x^i drawn from q^i) are tested in order with their
  own uniform; the first accepted one is kept; after each rejection
  p <- norm(max(0, p - q^i)); if none is accepted a token is drawn from the
  final residual.
* Section "Branch Resampling", "Branch Verification": the branch whose
  branch-point token is accepted is kept and the others are dropped, and
  ordinary speculative sampling continues along the kept branch (Appendix:
  Algorithm 1 runs only at branch points).

The walk generalises both to any token tree: at a node with several
children it runs Algorithm 1 over the children in ascending row order; with
one child it is the ordinary chain test.

Numeric contract (the HIP path follows the same one; only summation order
and exp ulps may differ):
  z_v = fl32(l_v * fl32(1/T)), M = max z, w_v = fl32(exp(fl32(z_v - M))),
  S = sum_v w_v in float64, p(v) = w_v / S in float64;
  T = 0 means p = one-hot at the lowest index of max l;
  accept iff float64(u) < p~(x) / float64(q(x))   (float64 division);
  residual r_v = max(0, p~(v) - q(v)) in float64, Z = sum r, p~ <- r / Z;
  Z <= 0 keeps p~ and raises FLAG_ZERO_RESIDUAL;
  draw: C_v = sum_{t<=v} p~(t) (float64, vocab order), W = C_{V-1},
  y = min{v : C_v > u * W}; zero-mass tokens are never drawn.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

from . import tree

FLAG_NONFINITE = 1        # a target row holds NaN or +Inf
FLAG_QZERO = 2            # a drafted token has q(x) == 0
FLAG_ZERO_RESIDUAL = 4    # a residual had no mass; p~ left unchanged


@dataclass
class RowStats:
    zmax: float       # max_v fl32(l_v / T)   (max l for T = 0)
    argmax: int       # lowest index of max l
    total: float      # sum_v fl32(exp(z_v - zmax)) in float64 (1.0 for T = 0)
    nonfinite: bool


def inv_temperature(T: float) -> np.float32:
    return np.float32(1.0) / np.float32(T)


def row_stats(logits_row, T: float) -> RowStats:
    """Statistics of one logits row.  A -inf logit is a masked token (zero
    probability); NaN or +inf make the row non-finite, and its total is NaN
    so that every later use of the row can see it."""
    l = np.asarray(logits_row, dtype=np.float32)
    nonfinite = bool(np.any(np.isnan(l) | (l == np.inf)))
    am = int(np.argmax(np.where(np.isnan(l), -np.inf, l)))
    if T > 0:
        z = l * inv_temperature(T)
        M = np.float32(np.max(np.where(np.isnan(z), -np.inf, z)))
        with np.errstate(invalid="ignore", over="ignore"):
            w = np.exp(z - M)
        S = math.fsum(w.astype(np.float64).tolist()) if not nonfinite else float("nan")
        return RowStats(float(M), am, S, nonfinite)
    return RowStats(float(l[am]), am, float("nan") if nonfinite else 1.0, nonfinite)


def target_probs(logits_row, T: float, st: RowStats | None = None) -> np.ndarray:
    """Target distribution p of one row as float64."""
    l = np.asarray(logits_row, dtype=np.float32)
    st = st or row_stats(l, T)
    if T > 0:
        z = l * inv_temperature(T)
        w = np.exp(z - np.float32(st.zmax))
        return w.astype(np.float64) / np.float64(st.total)
    p = np.zeros(l.shape[0], dtype=np.float64)
    p[st.argmax] = 1.0
    return p


def draw(weights: np.ndarray, u: float, trace: list | None = None, u_index: int = 0) -> int:
    """Inverse-CDF draw from non-negative float64 weights in vocab order."""
    w = np.asarray(weights, dtype=np.float64)
    C = np.cumsum(w)
    W = C[-1]
    if trace is not None:
        trace.append(("draw", u_index, C.copy(), float(W)))
    hit = np.nonzero(C > np.float64(u) * W)[0]
    if len(hit):
        return int(hit[0])
    pos = np.nonzero(w > 0)[0]
    return int(pos[-1]) if len(pos) else int(len(w) - 1)


@dataclass
class SelectResult:
    accepted: int | None          # index into the candidate list, or None
    p_tilde: np.ndarray           # distribution after the rejections
    flags: int = 0
    n_rejected: int = 0


def branch_select(p_tilde: np.ndarray, cand_tokens, cand_q, cand_u,
                  trace: list | None = None, cand_rows=None) -> SelectResult:
    """Algorithm 1 without its final draw: test candidates in order.

    cand_q[i] is the distribution candidate i was drawn from, cand_u[i] its
    uniform.  Returns the first accepted candidate (or None) and the
    residual distribution left after the rejections before it.
    """
    pt = np.asarray(p_tilde, dtype=np.float64)
    flags = 0
    nrej = 0
    for i, x in enumerate(cand_tokens):
        x = int(x)
        qrow = np.asarray(cand_q[i], dtype=np.float32)
        qx = np.float64(qrow[x])
        if qx == 0.0:
            flags |= FLAG_QZERO
        with np.errstate(divide="ignore", invalid="ignore"):
            ratio = np.float64(pt[x]) / qx
        if trace is not None:
            trace.append(("accept", int(cand_rows[i]) if cand_rows is not None else i, float(ratio)))
        if np.float64(cand_u[i]) < ratio:
            return SelectResult(i, pt, flags, nrej)
        nrej += 1
        r = np.maximum(0.0, pt - qrow.astype(np.float64))
        Z = math.fsum(r.tolist())
        if Z > 0.0:
            pt = r / np.float64(Z)
        else:
            flags |= FLAG_ZERO_RESIDUAL
    return SelectResult(None, pt, flags, nrej)


def select_branch(p_row: np.ndarray, cand_tokens, cand_q, u) -> tuple[int, int, int]:
    """Algorithm 1 in full: returns (accepted candidate index or -1, token,
    flags).  u[0..n-1] test the candidates, u[n] drives the final draw."""
    n = len(cand_tokens)
    res = branch_select(p_row, cand_tokens, cand_q, u[:n])
    if res.accepted is not None:
        return res.accepted, int(cand_tokens[res.accepted]), res.flags
    y = draw(res.p_tilde, float(u[n]))
    return -1, y, res.flags


@dataclass
class StepResult:
    n_accepted: int
    branch: int                 # ordinal of the kept root child, -1 if none
    next_token: int
    path: list = field(default_factory=list)   # rows root..last accepted
    flags: int = 0
    n_rejected: int = 0
    bonus: bool = False         # next_token drawn from p of a fully accepted leaf


def accept_resample(tokens, parents, logits, T: float, q, u, stats=None,
                    trace: list | None = None) -> StepResult:
    """Walk the token tree from the root (Algorithm 1 at every node, which is
    the chain test where a node has one child) and draw the next token."""
    tree.validate(parents)
    logits = np.asarray(logits, dtype=np.float32)
    N = len(parents)
    if stats is None:
        stats = [row_stats(logits[i], T) for i in range(N)]
    flags = 0
    if any(not math.isfinite(s.total) for s in stats):
        flags |= FLAG_NONFINITE
    node = 0
    path = [0]
    pt = target_probs(logits[0], T, stats[0])
    nrej = 0
    while True:
        kids = tree.children(parents, node)
        if not kids:
            y = draw(pt, float(u[0]), trace, 0)
            bonus = True
            break
        res = branch_select(pt, [tokens[c] for c in kids], [q[c] for c in kids],
                            [u[c] for c in kids], trace, kids)
        flags |= res.flags
        nrej += res.n_rejected
        if res.accepted is not None:
            node = kids[res.accepted]
            path.append(node)
            pt = target_probs(logits[node], T, stats[node])
            continue
        y = draw(res.p_tilde, float(u[0]), trace, 0)
        bonus = False
        break
    root_kids = tree.children(parents, 0)
    branch = root_kids.index(path[1]) if len(path) > 1 else -1
    return StepResult(len(path) - 1, branch, int(y), path, flags, nrej, bonus)
