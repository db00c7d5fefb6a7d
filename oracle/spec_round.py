"""Oracle of one whole SpecBranch round (test infrastructure only).

Algorithm 2 alternates a drafting phase and a verification phase; the
round here is one drafting phase followed by the verification phase that
consumes it, with the branch point chosen by confidence (Section "Branch
Resampling"):

1. drafting (drafting.draft_round): the draft, whose cache holds the
   committed prefix, scores the root (the last committed token) and drafts
   a chain x_1 .. x_c of confident tokens; the first unconfident draw (or
   the last allowed one) is the branch point x_b, drawn from q_b;
2. verification, while the draft spawns B candidates at x_b from q_b and
   extends each branch (the two run concurrently in the paper; here they
   are independent computations): the target scores the chain
   [root, x_1 .. x_c] on its own prefix cache, and the chain test of
   speculative sampling (Preliminaries; sampling.accept_resample over the
   chain, uniform u_walk[i] for x_i, u_walk[0] for a draw) accepts
   x_1 .. x_n;
3. n < c: the later drafts and every branch are dropped and the token is
   the residual draw at the first rejected position;
   n = c: no bonus token is drawn; Branch Speculative Sampling (Appendix,
   Algorithm 1) tests the candidates against p at row c -- the
   distribution of the position x_b occupies -- each with the q row it
   was drawn from (u_sel[i] for candidate i, u_sel[B] for the final draw);
   an accepted candidate's branch is kept, otherwise the token is the
   final residual draw (with B = 0 the token is the walk's draw from p at
   row c);
4. the target's cache keeps the root and x_1 .. x_n (rollback.kv_rollback
   over the walk's path); the draft's cache keeps the root, x_1 .. x_n and,
   with a kept branch, the branch's rows at depths 1 .. depth - 1, the
   ones whose keys and values the draft computed while extending it.

The committed tokens of the round are x_1 .. x_n and the token; with a kept
branch, its later drafts (depths 2 .. depth) are what the next verification
phase checks (Algorithm 2 stays in VERIFICATION).

Algorithm 2 tests a chain draft against its q row as drawn.  A draft stays
in the chain only when its own probability reaches epsilon, so a chain cut
by that test holds drafts drawn, in effect, from q restricted to the
confident tokens; with exact_chain each chain draft carries that
conditioned row instead, which keeps the committed tokens distributed as p
for any threshold (both forms are pinned by exact enumeration).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import decoder, drafting, rollback, sampling


@dataclass
class RoundResult:
    draft: drafting.DraftRound
    walk: sampling.StepResult      # the chain test over [root, x_1 .. x_c]
    n_trunk: int                   # accepted chain drafts
    kept: int                      # kept candidate, -1 if none
    token: int                     # the committed token after x_1 .. x_n
    flags: int
    logits: np.ndarray             # target logits of the chain rows
    draft_path: list               # draft tree rows the draft's cache keeps
    target_cache: tuple            # (K, V, new length) after the rollback
    draft_cache: tuple             # (K, V, new length) after the rollback

    @property
    def committed(self) -> list:
        return [int(t) for t in self.draft.tokens[1:1 + self.n_trunk]] + [self.token]


def uniforms_needed(k_max: int, depth: int, trunk_max: int) -> tuple[int, int, int]:
    """Lengths of u_draft, u_walk and u_sel."""
    return drafting.uniforms_needed(k_max, depth, trunk_max), trunk_max + 1, k_max + 1


def spec_round(tshape, tweights: dict, t_prefix_k, t_prefix_v, t_len: int,
               dshape, dweights: dict, d_prefix_k, d_prefix_v, d_len: int, root: int,
               k_max: int, mode: str, depth: int, T: float, u_draft, u_walk, u_sel,
               trunk_max: int = 1, epsilon: float = float("inf"), capacity: int | None = None,
               prec: str = "f64", trace: list | None = None,
               exact_chain: bool = False) -> RoundResult:
    """One round.  The prefix caches are [n_layers][n_kv][>= len][d]; the
    returned caches have `capacity` slots (default: prefix + every tree
    row).  With `trace`, every decision against a uniform is recorded
    (sampling.draw / branch_select events) with the uniform's index in the
    concatenation u_draft + u_walk + u_sel.  exact_chain: the chain drafts
    are tested against q conditioned on confidence (drafting.confident_row)."""
    nd, nw, ns = uniforms_needed(k_max, depth, trunk_max)
    u_walk = np.asarray(u_walk, dtype=np.float32)
    u_sel = np.asarray(u_sel, dtype=np.float32)
    assert len(u_walk) >= nw and len(u_sel) >= ns
    sub = [] if trace is not None else None

    def record(events, offset):
        if trace is not None:
            trace.extend((ev[0], offset + ev[1]) + tuple(ev[2:]) for ev in events)
            events.clear()

    # 1. drafting
    dr = drafting.draft_round(dshape, dweights, d_prefix_k, d_prefix_v, d_len, root, k_max, mode,
                              depth, T, u_draft, prec, trunk_max, epsilon, sub, exact_chain)
    record(sub, 0)
    c, B = dr.chain, dr.branches
    n_rows = len(dr.tokens)

    # 2. the target verifies the chain
    ctoks = dr.tokens[:c + 1]
    cpar = dr.parents[:c + 1]
    logits, kt, vt = decoder.tree_forward(tshape, tweights, t_prefix_k, t_prefix_v, t_len, ctoks,
                                          cpar, prec)
    walk = sampling.accept_resample(ctoks, cpar, logits, T, dr.q[:c + 1], u_walk[:c + 1], None,
                                    sub)
    record(sub, nd)

    # 3. the committed token
    flags = walk.flags
    kept, token = -1, walk.next_token
    n = walk.n_accepted
    if n == c and B > 0:
        cand = dr.tokens[c + 1:c + 1 + B]
        cq = dr.q[c + 1:c + 1 + B]
        p_c = sampling.target_probs(logits[c], T)
        res = sampling.branch_select(p_c, cand, cq, u_sel[:B], sub)
        flags |= res.flags
        if res.accepted is not None:
            kept, token = res.accepted, int(cand[res.accepted])
        else:
            token = sampling.draw(res.p_tilde, float(u_sel[B]), sub, B)
        record(sub, nd + nw)

    # 4. rollbacks
    cap = capacity if capacity is not None else max(t_len, d_len) + n_rows
    Kt, Vt = decoder.make_cache(tshape, t_prefix_k, t_prefix_v, t_len, cap)
    Kt, Vt = decoder.write_tree_kv(Kt, Vt, t_len, kt, vt)
    target_cache = rollback.kv_rollback(Kt, Vt, t_len, walk.path)
    # the draft's keys and values: rows up to depth - 1 of every branch (the
    # last depth's tokens were drawn but never scored)
    n_kv_rows = 1 + c + B * (depth - 1)
    _, kd, vd = decoder.tree_forward(dshape, dweights, d_prefix_k, d_prefix_v, d_len,
                                     dr.tokens[:n_kv_rows], dr.parents[:n_kv_rows], prec)
    dpath = list(range(n + 1))
    if kept >= 0:
        dpath += [c + 1 + (d - 1) * B + kept for d in range(1, depth)]
    Kd, Vd = decoder.make_cache(dshape, d_prefix_k, d_prefix_v, d_len, cap)
    Kd, Vd = decoder.write_tree_kv(Kd, Vd, d_len, kd, vd)
    draft_cache = rollback.kv_rollback(Kd, Vd, d_len, dpath)
    return RoundResult(dr, walk, n, kept, int(token), flags, logits, dpath, target_cache,
                       draft_cache)
