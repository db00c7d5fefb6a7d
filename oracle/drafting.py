"""Oracle of the draft side of one SpecBranch round (test infrastructure only).

``sample`` -- the draft's distribution at one row and the token drawn from
it.  q is the softmax of the draft's logits at temperature T (the same
definition as the target's p, Preliminaries, "Speculative Decoding"),
stored as float32 because that row is what verification later reads as q;
the token is the inverse-CDF draw (sampling.draw) over that float32 row with
the row's uniform.  T = 0: q is one-hot at the argmax (lowest index on
ties) and the token is the argmax.

``draft_round`` -- one drafting phase with its branch point right after the
root (Section "Branch Resampling", the drafting of Algorithm 2):
  1. the draft scores the root (the last committed token, not yet cached)
     on its prefix cache; x_b is drawn from that row's q with u[0];
  2. B sibling first tokens come from the same q by branching.candidates,
     with u[1 .. k_max], each carrying its own q row (reading R1);
  3. each branch then continues on its own prefix: its depth-d token
     (d = 2 .. depth) is drawn from the draft's distribution at its depth
     d - 1 row, with u[1 + k_max (d - 1) + i] for branch i.
The tree is depth-major: row 1 + (d - 1) B + i holds branch i's depth-d
token; its parent is row 0 at d = 1 and row - B after that.  Row i of the
returned q is the distribution token i was drawn from (row 0: the root's
distribution, the one x_b came from).  Every step scores the whole tree so
far with decoder.tree_forward; a row's logits do not depend on later rows.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import branching, decoder, sampling


def sample(logits_row, T: float, u: float):
    """(q float32 [V], token)."""
    q = sampling.target_probs(np.asarray(logits_row, dtype=np.float32), T).astype(np.float32)
    return q, sampling.draw(q.astype(np.float64), float(u))


@dataclass
class DraftRound:
    tokens: np.ndarray    # int32 [1 + B depth], row 0 the root
    parents: np.ndarray   # int32 [1 + B depth]
    q: np.ndarray         # float32 [1 + B depth][V]
    branches: int         # B
    x_b: int


def uniforms_needed(k_max: int, depth: int) -> int:
    return 1 + k_max * depth


def draft_round(shape, weights: dict, prefix_k, prefix_v, kv_len: int, root_token: int,
                k_max: int, mode: str, depth: int, T: float, u, prec: str = "f64") -> DraftRound:
    u = np.asarray(u, dtype=np.float32)
    assert depth >= 1 and len(u) >= uniforms_needed(k_max, depth)
    toks = [int(root_token)]
    parents = [-1]
    lg, _, _ = decoder.tree_forward(shape, weights, prefix_k, prefix_v, kv_len, toks, parents, prec)
    q_root, x_b = sample(lg[0], T, u[0])
    cand, rows = branching.candidates(q_root, x_b, k_max, mode, u[1:1 + k_max])
    B = len(cand)
    q = [q_root] + list(rows)
    toks += [int(t) for t in cand]
    parents += [0] * B
    for d in range(2, depth + 1 if B else 0):
        lg, _, _ = decoder.tree_forward(shape, weights, prefix_k, prefix_v, kv_len, toks, parents,
                                        prec)
        for i in range(B):
            r = 1 + (d - 2) * B + i
            qi, t = sample(lg[r], T, u[1 + k_max * (d - 1) + i])
            toks.append(t)
            parents.append(r)
            q.append(qi)
    return DraftRound(np.asarray(toks, dtype=np.int32), np.asarray(parents, dtype=np.int32),
                      np.stack(q).astype(np.float32), B, int(x_b))
