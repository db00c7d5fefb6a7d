"""Oracle of the draft side of one SpecBranch round (test infrastructure only).

``sample`` -- the draft's distribution at one row and the token drawn from
it.  q is the softmax of the draft's logits at temperature T (the same
definition as the target's p, Preliminaries, "Speculative Decoding"),
stored as float32 because that row is what verification later reads as q;
the token is the inverse-CDF draw (sampling.draw) over that float32 row with
the row's uniform.  T = 0: q is one-hot at the argmax (lowest index on
ties) and the token is the argmax.

``draft_round`` -- one drafting phase (Section "Branch Resampling", the
drafting of Algorithm 2), with the branch point at the draft's first
unconfident token:
  1. the draft scores the root (the last committed token, not yet cached)
     on its prefix cache and drafts a chain: x_t (t = 1, 2, ...) is drawn
     from the distribution at row t - 1 with u[t - 1].  The branch point is
     the first x_t whose own probability q(x_t) is below the confidence
     threshold epsilon (both float32), or x_trunk_max; the confident tokens
     before it, c = t - 1 of them, stay in the tree as a chain (rows 1 .. c);
  2. x_b = that token sets B, and B sibling first tokens come from the
     distribution it was drawn from by branching.candidates, with
     u[trunk_max .. trunk_max + k_max - 1], each carrying its own q row
     (reading R1);
  3. each branch then continues on its own prefix: its depth-d token
     (d = 2 .. depth) is drawn from the draft's distribution at its depth
     d - 1 row, with u[trunk_max + k_max (d - 1) + i] for branch i.
trunk_max = 1 puts the branch point right after the root (x_b = x_1).
The branches are depth-major: row c + 1 + (d - 1) B + i holds branch i's
depth-d token; its parent is row c at d = 1 and row - B after that.  Row i
of the returned q is the distribution token i was drawn from, and row 0
(the root, which verification does not test) holds the branch position's
distribution, the one x_b came from.  Every step scores the whole tree so
far with decoder.tree_forward; a row's logits do not depend on later rows.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

from . import branching, decoder, sampling


def sample(logits_row, T: float, u: float, trace: list | None = None, u_index: int = 0):
    """(q float32 [V], token).  With `trace`, the draw is recorded as
    sampling.draw records it, under uniform index u_index."""
    q = sampling.target_probs(np.asarray(logits_row, dtype=np.float32), T).astype(np.float32)
    return q, sampling.draw(q.astype(np.float64), float(u), trace, u_index)


@dataclass
class DraftRound:
    tokens: np.ndarray    # int32 [1 + c + B depth], row 0 the root
    parents: np.ndarray   # int32, same length
    q: np.ndarray         # float32 [rows][V]
    branches: int         # B
    x_b: int
    chain: int = 0        # c, the confident drafts before the branch point


def uniforms_needed(k_max: int, depth: int, trunk_max: int = 1) -> int:
    return trunk_max + k_max * depth


def confident_row(q_row, epsilon: float) -> np.ndarray:
    """q conditioned on confidence: q(v) / q(C) on C = {v : q(v) >= epsilon}
    (float32 comparisons, q(C) the float64 sum of the float32 values), zero
    elsewhere, stored as float32.  A chain draft was kept because its own
    probability reached epsilon, so it was in effect drawn from this row."""
    q = np.asarray(q_row, dtype=np.float32)
    keep = q >= np.float32(epsilon)
    mass = math.fsum(q[keep].astype(np.float64).tolist())
    out = np.zeros(len(q), dtype=np.float32)
    if mass > 0.0:
        out[keep] = (q[keep].astype(np.float64) / mass).astype(np.float32)
    return out


def draft_round(shape, weights: dict, prefix_k, prefix_v, kv_len: int, root_token: int,
                k_max: int, mode: str, depth: int, T: float, u, prec: str = "f64",
                trunk_max: int = 1, epsilon: float = float("inf"),
                trace: list | None = None, exact_chain: bool = False) -> DraftRound:
    """With `trace`, every draw is recorded (sampling.draw's events) under
    the index of its uniform in u.  With `exact_chain`, a chain draft carries
    confident_row(q, epsilon) as the row its test divides by, instead of q
    (the variant that keeps the round exactly lossless when the chain's
    length depends on the drafts' own probabilities)."""
    u = np.asarray(u, dtype=np.float32)
    assert depth >= 1 and trunk_max >= 1
    assert len(u) >= uniforms_needed(k_max, depth, trunk_max)
    eps = np.float32(epsilon)
    toks = [int(root_token)]
    parents = [-1]
    q = [None]
    for t in range(1, trunk_max + 1):
        lg, _, _ = decoder.tree_forward(shape, weights, prefix_k, prefix_v, kv_len, toks, parents,
                                        prec)
        q_t, x_t = sample(lg[t - 1], T, u[t - 1], trace, t - 1)
        if t == trunk_max or q_t[x_t] < eps:
            q_b, x_b = q_t, x_t
            break
        toks.append(x_t)
        parents.append(t - 1)
        q.append(confident_row(q_t, epsilon) if exact_chain else q_t)
    c = len(toks) - 1
    q[0] = q_b
    u0 = trunk_max
    sub = [] if trace is not None else None
    cand, rows = branching.candidates(q_b, x_b, k_max, mode, u[u0:u0 + k_max], sub)
    if trace is not None:
        trace += [(ev[0], u0 + ev[1]) + tuple(ev[2:]) for ev in sub]
    B = len(cand)
    q += list(rows)
    toks += [int(t) for t in cand]
    parents += [c] * B
    for d in range(2, depth + 1 if B else 0):
        lg, _, _ = decoder.tree_forward(shape, weights, prefix_k, prefix_v, kv_len, toks, parents,
                                        prec)
        for i in range(B):
            r = c + 1 + (d - 2) * B + i
            ui = u0 + k_max * (d - 1) + i
            qi, t = sample(lg[r], T, u[ui], trace, ui)
            toks.append(t)
            parents.append(r)
            q.append(qi)
    return DraftRound(np.asarray(toks, dtype=np.int32), np.asarray(parents, dtype=np.int32),
                      np.stack(q).astype(np.float32), B, int(x_b), c)
