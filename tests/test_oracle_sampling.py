"""Pins of the oracle accept / select / resample walk (CPU only).

* Hand-worked golden cases (tests/golden/accept_cases.txt).
* Row statistics against scipy's softmax; T = 0 reduces to argmax with
  lowest-index ties.
* Exact enumeration over the uniforms (tests/walk_enum.py):
  - the first emitted token is distributed exactly as the target p for
    i.i.d. candidates, candidates drawn without replacement and
    deterministic top-k with one-hot q rows, and NOT for top-k candidates
    tested against one shared q (the reading of the candidate rows that the
    paper's Algorithm 1 needs: each candidate is tested against the
    distribution it was drawn from);
  - the whole step (Algorithm 1 at the branch point, chain speculative
    sampling below it, residual or bonus draw) is lossless: emitted tokens
    continued by the target reproduce the target's own sequence law;
  - a chain with constant acceptance ratio alpha has the truncated
    geometric accepted length of Section "Theoretical Speedup" and the mean
    of Lemma 1;
  - along a fixed chain P(n >= j) = prod_{i<=j} min(1, p_i/q_i).
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
from scipy.special import softmax

from oracle import decoder, sampling
from paper_2506_01979_amd import synth
from walk_enum import enumerate_outcomes

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "accept_cases.txt")


def golden_cases():
    with open(GOLDEN) as f:
        return [json.loads(l) for l in f if l.strip() and not l.startswith("#")]


@pytest.mark.parametrize("case", golden_cases(), ids=lambda c: c["name"])
def test_golden_select(case):
    p = np.asarray(case["p"], dtype=np.float64)
    q = [np.asarray(r, dtype=np.float32) for r in case["q"]]
    acc, tok, _ = sampling.select_branch(p, case["x"], q, case["u"])
    assert acc == case["accepted"]
    assert tok == case["token"]


def test_row_stats_and_probs_match_softmax():
    g = np.random.default_rng(0)
    for T in (1.0, 0.7, 2.5):
        l = (g.standard_normal(3000) * 4).astype(np.float32)
        st = sampling.row_stats(l, T)
        p = sampling.target_probs(l, T, st)
        assert abs(p.sum() - 1.0) < 1e-12
        ref = softmax(l.astype(np.float64) / T)
        # fl32(l/T) and fl32(z - M) carry about |z| * 2^-24 absolute error
        assert np.max(np.abs(p - ref) / ref) < 1e-5
        assert st.argmax == int(np.argmax(l))


def test_greedy_is_argmax_lowest_index():
    l = np.array([0.5, 2.0, -1.0, 2.0, 1.0], dtype=np.float32)
    st = sampling.row_stats(l, 0.0)
    assert st.argmax == 1
    p = sampling.target_probs(l, 0.0, st)
    assert list(p) == [0, 1, 0, 0, 0]
    # greedy chain: accept iff the draft is the argmax, emit the argmax
    par = [-1, 0, 1]
    logits = np.stack([l, l, l])
    q = np.full((3, 5), 0.2, dtype=np.float32)
    for toks, n_acc in (([0, 1, 1], 2), ([0, 1, 3], 1), ([0, 3, 1], 0)):
        r = sampling.accept_resample(toks, par, logits, 0.0, q, np.full(3, 0.999, np.float32))
        assert r.n_accepted == n_acc and r.next_token == 1


def test_flags():
    par = [-1, 0]
    logits = np.zeros((2, 4), dtype=np.float32)
    q = np.zeros((2, 4), dtype=np.float32)
    q[1] = [0.0, 0.5, 0.5, 0.0]
    r = sampling.accept_resample([0, 0], par, logits, 1.0, q, np.array([0.5, 0.5], np.float32))
    assert r.flags & sampling.FLAG_QZERO and r.n_accepted == 1   # p/0 = inf
    logits[1, 2] = np.nan
    r = sampling.accept_resample([0, 1], par, logits, 1.0, q, np.array([0.5, 0.5], np.float32))
    assert r.flags & sampling.FLAG_NONFINITE


def test_zero_residual_flag():
    p = np.array([0.5, 0.5, 0.0], dtype=np.float64)
    q = [np.array([0.5, 0.5, 0.0], dtype=np.float32)]
    res = sampling.branch_select(p, [0], q, [0.999])   # ratio 1: rejected only as u >= 1
    assert res.accepted == 0
    q = [np.array([0.25, 0.75, 0.0], dtype=np.float32)]
    res = sampling.branch_select(np.array([0.0, 1.0, 0.0]), [1], q, [0.9])
    assert res.accepted == 0
    # a (non-normalised) q that dominates p everywhere leaves no residual
    # mass after a rejection: p~ is kept and the flag raised
    p = np.array([0.25, 0.5, 0.25])
    res = sampling.branch_select(p, [1], [np.array([0.5, 1.0, 0.5], np.float32)], [0.9])
    assert res.accepted is None
    assert res.flags & sampling.FLAG_ZERO_RESIDUAL
    assert np.array_equal(res.p_tilde, p)


# ----------------------------------------------------------------------------
# exact enumeration
# ----------------------------------------------------------------------------

def dyadic(prob: np.ndarray, bits: int = 20) -> np.ndarray:
    """float32 distribution with entries k / 2^bits summing exactly to 1, so
    the draw weights and the q rows the walk reads are the same numbers."""
    k = np.maximum(1, np.round(prob * 2 ** bits)).astype(np.int64)
    k[np.argmax(k)] += 2 ** bits - k.sum()
    return (k / 2.0 ** bits).astype(np.float32)


def q_exact():
    g = np.random.default_rng(11)
    V = 16
    q = dyadic(softmax(g.standard_normal(V) * 1.0))
    p = softmax(g.standard_normal(V) * 1.3)
    return p, q


def _enum_first_token(p, cand_sets, n_cand):
    V = len(p)
    parents = [-1] + [0] * n_cand
    logits = np.zeros((1 + n_cand, V), dtype=np.float32)
    logits[0] = np.log(p).astype(np.float32)
    p_used = sampling.target_probs(logits[0], 1.0)
    dist = np.zeros(V)
    for wgt, toks, qrows in cand_sets:
        tokens = [0] + [int(t) for t in toks]
        q = np.zeros((1 + n_cand, V), dtype=np.float32)
        q[1:] = qrows

        def run(u, tokens=tokens, q=q):
            tr = []
            return sampling.accept_resample(tokens, parents, logits, 1.0, q, u, trace=tr), tr

        def project(r, tokens=tokens):
            return tokens[r.path[1]] if r.n_accepted else r.next_token

        def relevant(r, tr):
            # the first token is fixed by the root's accept tests; the draw
            # that follows matters only when every candidate was rejected
            return len(tr) - 1 if r.n_accepted else len(tr)

        out = enumerate_outcomes(run, 1 + n_cand, project, relevant)
        for v, pr in out.items():
            dist[v] += wgt * pr
    return p_used, dist


def iid_sets(q, B):
    V = len(q)
    qd = q.astype(np.float64)
    for toks in itertools.product(range(V), repeat=B):
        yield float(np.prod(qd[list(toks)])), toks, np.stack([q] * B)


def wo_replacement_sets(q, B):
    V = len(q)
    qd = q.astype(np.float64)
    for toks in itertools.permutations(range(V), B):
        w = 1.0
        rows = []
        avail = qd.copy()
        for t in toks:
            row = avail / avail.sum()
            w *= row[t]
            rows.append(row.astype(np.float32))
            avail[t] = 0.0
        yield w, toks, np.stack(rows)


def topk_sets(q, B, onehot: bool):
    toks = list(np.argsort(-q, kind="stable")[:B])
    if onehot:
        rows = np.zeros((B, len(q)), dtype=np.float32)
        rows[np.arange(B), toks] = 1.0
    else:
        rows = np.stack([q] * B)
    yield 1.0, toks, rows


@pytest.mark.parametrize("kind", ["iid", "without_replacement", "topk_onehot"])
def test_first_token_is_target_distributed(kind):
    p, q = q_exact()
    B = 3
    sets = {"iid": iid_sets(q, B), "without_replacement": wo_replacement_sets(q, B),
            "topk_onehot": topk_sets(q, B, True)}[kind]
    p_used, dist = _enum_first_token(p, sets, B)
    # conditional rows without replacement are rounded to float32, so the
    # walk's q and the draw law differ by ~1e-8 there
    tol = 1e-6 if kind == "without_replacement" else 1e-9
    assert abs(dist.sum() - 1.0) < tol
    assert np.max(np.abs(dist - p_used)) < tol


def test_topk_with_shared_q_is_not_lossless():
    p, q = q_exact()
    p_used, dist = _enum_first_token(p, topk_sets(q, 3, False), 3)
    assert abs(dist.sum() - 1.0) < 1e-9
    assert np.max(np.abs(dist - p_used)) > 1e-3


def _const_ratio_chain(alpha, gamma, V=4):
    """Chain of gamma drafts whose tested tokens all have p/q = alpha."""
    parents = list(range(-1, gamma))
    tokens = [0] + [1] * gamma
    q = np.zeros((gamma + 1, V), dtype=np.float32)
    q[1:] = [0.1, 0.5, 0.2, 0.2]
    p = np.array([0.3, 0.5 * alpha, 0.2, 0.5 - 0.5 * alpha])
    logits = np.tile(np.log(p).astype(np.float32), (gamma + 1, 1))
    return parents, tokens, q, logits


@pytest.mark.parametrize("alpha,gamma", [(0.3, 4), (0.6, 8), (0.9, 5)])
def test_truncated_geometric_and_lemma1(alpha, gamma):
    parents, tokens, q, logits = _const_ratio_chain(alpha, gamma)
    ratio = sampling.target_probs(logits[1], 1.0)[1] / np.float64(q[1, 1])

    def run(u):
        tr = []
        return sampling.accept_resample(tokens, parents, logits, 1.0, q, u, trace=tr), tr

    dist = enumerate_outcomes(run, gamma + 1, lambda r: r.n_accepted,
                              lambda r, tr: sum(1 for e in tr if e[0] == "accept"))
    a = ratio
    for kk in range(gamma + 1):
        want = (1 - a) * a ** kk if kk < gamma else a ** gamma
        assert abs(dist.get(kk, 0.0) - want) < 1e-12
    mean = sum(kk * pr for kk, pr in dist.items())
    assert abs(mean - a * (1 - a ** gamma) / (1 - a)) < 1e-12
    assert abs(a - alpha) < 1e-6


def test_chain_acceptance_product():
    g = np.random.default_rng(5)
    V, gamma = 12, 5
    parents = list(range(-1, gamma))
    logits = (g.standard_normal((gamma + 1, V)) * 2).astype(np.float32)
    q = softmax(g.standard_normal((gamma + 1, V)), axis=-1).astype(np.float32)
    tokens = [0] + list(g.integers(0, V, gamma))

    def run(u):
        tr = []
        return sampling.accept_resample(tokens, parents, logits, 1.0, q, u, trace=tr), tr

    dist = enumerate_outcomes(run, gamma + 1, lambda r: r.n_accepted,
                              lambda r, tr: sum(1 for e in tr if e[0] == "accept"))
    beta = [min(1.0, sampling.target_probs(logits[i - 1], 1.0)[tokens[i]] / float(q[i, tokens[i]]))
            for i in range(1, gamma + 1)]
    for j in range(gamma + 1):
        tail = sum(pr for kk, pr in dist.items() if kk >= j)
        assert abs(tail - float(np.prod(beta[:j]))) < 1e-12


# ----------------------------------------------------------------------------
# whole-step losslessness on a tiny model
# ----------------------------------------------------------------------------

V4 = synth.Shape("exact_v4", 1, 64, 2, 2, 32, 172, 4, "f32")


def test_whole_step_is_lossless():
    """B = 2 branches x k = 2 drafts, V = 4: for every length-3 sequence t,
    sum over emitted prefixes s of t of P_step(s) * p_target(rest of t | s)
    equals p_target(t)."""
    shape = V4
    W = synth.model_weights(shape)
    P = 6
    B, k = 2, 2
    ptoks = synth.prefix_tokens(shape.vocab, P)
    _, Kp, Vp = decoder.prefill(shape, W, ptoks[:-1], "f64")
    parents = synth.branch_parents(B, k)   # [-1, 0, 1, 0, 3]
    Vv = shape.vocab
    g = np.random.default_rng(2)
    q1 = dyadic(softmax(g.standard_normal(Vv)))
    q2 = dyadic(softmax(g.standard_normal(Vv)))

    # target conditionals p(. | prefix + s) for every s of length <= k
    cond = {}
    for L in range(0, k + 1):
        for s in itertools.product(range(Vv), repeat=L):
            lg, _, _ = decoder.tree_forward(shape, W, Kp, Vp, P - 1, [ptoks[-1], *s],
                                            synth.chain_parents(L + 1), "f64")
            cond[s] = sampling.target_probs(lg[-1].astype(np.float32), 1.0)

    def seq_prob(ctx, rest):
        pr = 1.0
        for t in rest:
            pr *= cond[tuple(ctx)][t]
            ctx = list(ctx) + [t]
        return pr

    step = {}   # emitted sequence -> probability
    for x1, x2, c1, c2 in itertools.product(range(Vv), repeat=4):
        wgt = float(q1[x1]) * float(q1[x2]) * float(q2[c1]) * float(q2[c2])
        tokens = [int(ptoks[-1]), x1, c1, x2, c2]
        lg, _, _ = decoder.tree_forward(shape, W, Kp, Vp, P - 1, tokens, parents, "f64")
        lg = lg.astype(np.float32)
        q = np.zeros((5, Vv), dtype=np.float32)
        q[1] = q[3] = q1
        q[2] = q[4] = q2

        def run(u, tokens=tokens, lg=lg, q=q):
            tr = []
            return sampling.accept_resample(tokens, parents, lg, 1.0, q, u, trace=tr), tr

        def project(r, tokens=tokens):
            return tuple(tokens[i] for i in r.path[1:]) + (r.next_token,)

        for s, pr in enumerate_outcomes(run, 5, project).items():
            step[s] = step.get(s, 0.0) + wgt * pr
    assert abs(sum(step.values()) - 1.0) < 1e-9
    worst = 0.0
    for t in itertools.product(range(Vv), repeat=k + 1):
        lhs = sum(pr * seq_prob(list(s), t[len(s):]) for s, pr in step.items()
                  if t[:len(s)] == s)
        rhs = seq_prob([], t)
        worst = max(worst, abs(lhs - rhs))
    assert worst < 1e-9


def test_minus_inf_logit_is_a_masked_token():
    """A -inf logit is a token with zero probability: it carries no mass in
    the row total, is never drawn (whatever the uniform), is never accepted
    as a draft, and the remaining tokens keep the softmax of the finite
    logits.  The row stays finite (no flag)."""
    l = np.array([0.3, -np.inf, 1.2, -np.inf, -0.7, 0.0], dtype=np.float32)
    fin = np.isfinite(l)
    st = sampling.row_stats(l, 1.0)
    assert not st.nonfinite
    w = np.exp(l[fin] - np.float32(1.2)).astype(np.float64)   # fl32(exp(fl32(z - M)))
    assert abs(st.total - w.sum()) < 1e-12
    p = sampling.target_probs(l, 1.0, st)
    assert np.all(p[~fin] == 0.0)
    assert abs(p.sum() - 1.0) < 1e-12
    ref = np.exp(l[fin].astype(np.float64)) / np.exp(l[fin].astype(np.float64)).sum()
    assert np.max(np.abs(p[fin] - ref)) < 1e-6
    # never drawn, over a fine grid of uniforms including both ends
    for u in np.concatenate([np.linspace(0.0, 1.0 - 2**-24, 4097), [0.0, 1.0 - 2**-24]]):
        assert fin[sampling.draw(p, float(u))]
    # a draft of a masked token is never accepted (p = 0 < u for every u,
    # and u = 0 is not < 0), and the emitted token is a finite-logit one
    par = [-1, 0]
    logits = np.stack([l, l])
    q = np.full((2, 6), 1.0 / 6.0, dtype=np.float32)
    for u1 in (0.0, 0.5, 1.0 - 2**-24):
        r = sampling.accept_resample([0, 1], par, logits, 1.0, q, np.array([0.3, u1], np.float32))
        assert r.n_accepted == 0 and fin[r.next_token] and r.flags == 0
    # greedy (T = 0) ignores -inf as well
    st0 = sampling.row_stats(l, 0.0)
    assert st0.argmax == 2 and not st0.nonfinite
