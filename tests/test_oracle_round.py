"""Pins of the whole-round oracle (oracle.spec_round, Algorithm 2).

* The round's outcome equals the pinned tree walk (sampling.accept_resample,
  itself pinned by exact enumeration) run on the tree "chain, then the
  candidates as children of the chain's last row", with the walk's
  uniforms wired to the round's: the chain test, the rejection draw and
  Algorithm 1 at the branch point compose as the walk composes them.
* Exact enumeration over every uniform of a round (drafting and
  verification) on a four-token vocabulary: the first committed token is
  distributed as the target's p at the root, and the second, given the
  first, as p after it -- the losslessness of speculative sampling
  (Preliminaries) and of Algorithm 1 -- for every branching mode, whenever
  the chain's length does not depend on the drafted values (trunk_max = 1,
  or confidence threshold 0).  A chain cut by the confidence of the
  drafted token itself is tested against the unconditioned q row, as
  Algorithm 2 writes the test; enumeration shows the resulting deviation
  from p, which the test records.
* After the round each cache holds exactly what a fresh prefill of the
  kept tokens computes: the target's the prefix, root and accepted drafts;
  the draft's the same plus the kept branch's scored rows.
* Greedy (T = 0) rounds reproduce the target's greedy decoding.
"""
import numpy as np
import pytest

from oracle import branching, decoder, sampling, spec_round
from paper_2506_01979_amd import synth
from walk_enum import enumerate_outcomes


def models(name, P, seed=2):
    sh = synth.SHAPES[name]
    Wt, Wd = synth.model_weights(sh, 0), synth.model_weights(sh, 1)
    ptoks = synth.prefix_tokens(sh.vocab, P + 1, seed)
    _, Kt, Vt = decoder.prefill(sh, Wt, ptoks[:-1])
    _, Kd, Vd = decoder.prefill(sh, Wd, ptoks[:-1])
    return sh, Wt, Wd, ptoks, Kt, Vt, Kd, Vd


def run_round(m, k_max, mode, depth, T, u_d, u_w, u_s, trunk, eps, trace=None, exact=False):
    sh, Wt, Wd, ptoks, Kt, Vt, Kd, Vd = m
    P = len(ptoks) - 1
    return spec_round.spec_round(sh, Wt, Kt, Vt, P, sh, Wd, Kd, Vd, P, int(ptoks[-1]), k_max, mode,
                                 depth, T, u_d, u_w, u_s, trunk, eps, trace=trace,
                                 exact_chain=exact)


@pytest.fixture
def memo_forward(monkeypatch):
    """Enumeration re-runs a round thousands of times on a handful of token
    trees: reuse each tree's forward."""
    orig = decoder.tree_forward
    cache = {}

    def fwd(shape, weights, pk, pv, kv_len, tokens, parents, mode="f64", hidden=None):
        key = (id(weights), kv_len, tuple(int(t) for t in tokens),
               tuple(int(p) for p in parents), mode)
        if hidden is not None:
            return orig(shape, weights, pk, pv, kv_len, tokens, parents, mode, hidden)
        if key not in cache:
            cache[key] = orig(shape, weights, pk, pv, kv_len, tokens, parents, mode)
        return cache[key]

    monkeypatch.setattr(decoder, "tree_forward", fwd)


WALK_CASES = [(mode, seed, trunk, eps) for mode in branching.MODES for seed in range(12)
              for trunk, eps in ((1, float("inf")), (4, 0.08))]


def test_round_is_the_tree_walk_over_chain_and_candidates():
    m = models("exact", 8)
    V = m[0].vocab
    k_max, depth, T = 4, 3, 0.25
    kinds = set()
    for mode, seed, trunk, eps in WALK_CASES:
        nd, nw, ns = spec_round.uniforms_needed(k_max, depth, trunk)
        u = synth.uniforms(nd + nw + ns, seed=100 + seed)
        u_d, u_w, u_s = u[:nd], u[nd:nd + nw].copy(), u[nd + nw:].copy()
        r = run_round(m, k_max, mode, depth, T, u_d, u_w, u_s, trunk, eps)
        c, B = r.draft.chain, r.draft.branches
        # one uniform drives the final draw in both: the walk's u[0]
        u_w[0] = u_s[B]
        r = run_round(m, k_max, mode, depth, T, u_d, u_w, u_s, trunk, eps)
        n = 1 + c + B
        toks, par, q = r.draft.tokens[:n], r.draft.parents[:n], r.draft.q[:n]
        # the candidates' logits rows are never read on a kept candidate but
        # for its bonus draw, which the round does not make
        logits = np.vstack([r.logits, np.zeros((B, V), dtype=r.logits.dtype)])
        u_t = np.concatenate([u_w[:c + 1], u_s[:B]])
        w = sampling.accept_resample(toks, par, logits, T, q, u_t)
        if len(w.path) == c + 2:
            kinds.add("kept")
            assert (r.n_trunk, r.kept, r.token) == (c, w.path[-1] - c - 1, int(toks[w.path[-1]]))
        else:
            kinds.add("chain rejected" if w.n_accepted < c else "candidates rejected")
            assert (r.n_trunk, r.kept, r.token) == (w.n_accepted, -1, w.next_token)
        assert r.flags == w.flags
        assert r.walk.path == list(range(r.n_trunk + 1))
    assert kinds == {"kept", "chain rejected", "candidates rejected"}


def enumerate_round(m, k_max, mode, depth, T, trunk, eps, exact=False):
    nd, nw, ns = spec_round.uniforms_needed(k_max, depth, trunk)

    def run(u):
        tr = []
        r = run_round(m, k_max, mode, depth, T, u[:nd], u[nd:nd + nw], u[nd + nw:], trunk, eps,
                      tr, exact)
        return r, tr

    out = enumerate_outcomes(run, nd + nw + ns, lambda r: tuple(r.committed[:2]))
    sh, Wt, _, ptoks, Kt, Vt, _, _ = m
    P, V = len(ptoks) - 1, sh.vocab
    root = int(ptoks[-1])
    e1, e12 = np.zeros(V), np.zeros((V, V))
    for k, pr in out.items():
        e1[k[0]] += pr
        if len(k) > 1:
            e12[k[0], k[1]] += pr
    lg, _, _ = decoder.tree_forward(sh, Wt, Kt, Vt, P, [root], [-1])
    err1 = np.abs(e1 - sampling.target_probs(lg[0], T)).max()
    err2 = 0.0
    for a in range(V):
        if e12[a].sum() > 0:
            lg, _, _ = decoder.tree_forward(sh, Wt, Kt, Vt, P, [root, a], [-1, 0])
            err2 = max(err2, np.abs(e12[a] / e12[a].sum() - sampling.target_probs(lg[1], T)).max())
    return abs(sum(out.values()) - 1.0), err1, err2, e12.sum()


# box midpoints are rounded to float32 uniforms, which moves a draw's
# outcome on boxes narrower than 2^-24: a few 1e-9 of probability
ENUM_TOL = 1e-7


@pytest.mark.parametrize("mode", branching.MODES)
def test_round_first_token_is_the_target_distribution(memo_forward, mode):
    m = models("enum", 4)
    vol, err1, _, _ = enumerate_round(m, 4, mode, 1, 0.3, 1, float("inf"))
    assert vol < 1e-12 and err1 < ENUM_TOL


@pytest.mark.parametrize("mode", branching.MODES)
def test_round_with_a_fixed_length_chain_is_lossless(memo_forward, mode):
    # threshold 0: every draft is confident, the chain always holds
    # trunk_max - 1 = 1 token and the branch point is the second position
    m = models("enum", 4)
    vol, err1, err2, p2 = enumerate_round(m, 3, mode, 1, 0.3, 2, 0.0)
    assert vol < 1e-12 and err1 < ENUM_TOL and err2 < ENUM_TOL
    assert p2 > 0.1                            # the second position is reached


def test_confidence_gated_chain_deviates_from_the_target(memo_forward):
    # a drafted token stays in the chain only when q(x) >= epsilon, so the
    # chain's tokens follow q restricted to the confident tokens while the
    # test divides by the unconditioned q(x): the first token's law moves
    # away from p (here by 0.09 on the largest entry)
    m = models("enum", 4)
    vol, err1, _, _ = enumerate_round(m, 3, "topk", 1, 0.3, 3, 0.2)
    assert vol < 1e-12 and 0.05 < err1 < 0.15


# a chain of 3 accepted and a kept branch; a chain of 2 rejected at its
# second token; no chain and a kept branch (the second candidate); no chain
# and every candidate rejected
@pytest.mark.parametrize("mode", branching.MODES)
@pytest.mark.parametrize("eps", [0.2, 0.35])
def test_conditioned_chain_is_lossless_at_any_threshold(memo_forward, mode, eps):
    # each chain draft tested against q conditioned on confidence: the first
    # and second committed tokens follow p exactly, with the chain's length
    # set by the drafts' own probabilities
    m = models("enum", 4)
    vol, err1, err2, p2 = enumerate_round(m, 3, mode, 1, 0.3, 3, eps, exact=True)
    assert vol < 1e-12 and err1 < ENUM_TOL and err2 < ENUM_TOL
    assert p2 > 0.02                           # the second position is reached


def test_confident_row_is_q_restricted_and_renormalised():
    q = np.array([0.5, 0.05, 0.3, 0.15], dtype=np.float32)
    from oracle import drafting
    r = drafting.confident_row(q, 0.15)
    assert r.dtype == np.float32
    np.testing.assert_allclose(r, [0.5 / 0.95, 0.0, 0.3 / 0.95, 0.15 / 0.95], rtol=1e-7)
    assert np.all(drafting.confident_row(q, 0.9) == 0.0)
    np.testing.assert_allclose(drafting.confident_row(q, 0.0), q / q.astype(np.float64).sum(),
                               rtol=1e-7)


ROLLBACK_CASES = [("wor", 9, 6, 0.08), ("iid", 7, 6, 0.08), ("topk", 1, 1, float("inf")),
                  ("topk", 3, 1, float("inf"))]


@pytest.mark.parametrize("mode,seed,trunk,eps", ROLLBACK_CASES)
def test_round_caches_equal_a_fresh_prefill(mode, seed, trunk, eps):
    m = models("exact", 8)
    sh, Wt, Wd, ptoks = m[:4]
    P = len(ptoks) - 1
    k_max, depth, T = 4, 4, 0.25
    nd, nw, ns = spec_round.uniforms_needed(k_max, depth, trunk)
    u = synth.uniforms(nd + nw + ns, seed=seed)
    r = run_round(m, k_max, mode, depth, T, u[:nd], u[nd:nd + nw], u[nd + nw:], trunk, eps)
    Kt, Vt, lt = r.target_cache
    Kd, Vd, ld = r.draft_cache
    kept_t = list(ptoks) + [int(t) for t in r.draft.tokens[1:1 + r.n_trunk]]
    assert lt == len(kept_t)
    _, K, V = decoder.prefill(sh, Wt, kept_t)
    np.testing.assert_allclose(Kt[:, :, :lt], K, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(Vt[:, :, :lt], V, rtol=1e-10, atol=1e-12)
    kept_d = list(ptoks[:-1]) + [int(r.draft.tokens[j]) for j in r.draft_path]
    assert ld == len(kept_d)
    if r.kept >= 0:
        assert len(r.draft_path) == r.n_trunk + depth and r.draft_path[r.n_trunk + 1:][:1] == \
            [1 + r.draft.chain + r.kept]
    _, K, V = decoder.prefill(sh, Wd, kept_d)
    np.testing.assert_allclose(Kd[:, :, :ld], K, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(Vd[:, :, :ld], V, rtol=1e-10, atol=1e-12)


def test_rollback_cases_cover_kept_and_dropped_branches():
    m = models("exact", 8)
    seen = set()
    for mode, seed, trunk, eps in ROLLBACK_CASES:
        nd, nw, ns = spec_round.uniforms_needed(4, 4, trunk)
        u = synth.uniforms(nd + nw + ns, seed=seed)
        r = run_round(m, 4, mode, 4, 0.25, u[:nd], u[nd:nd + nw], u[nd + nw:], trunk, eps)
        seen.add((r.kept >= 0, r.draft.chain > 0, r.n_trunk < r.draft.chain))
    assert seen == {(True, True, False), (False, True, True), (True, False, False),
                    (False, False, False)}


@pytest.mark.parametrize("trunk,eps", [(1, float("inf")), (5, 0.5), (5, 0.0)])
def test_greedy_round_reproduces_greedy_decoding(trunk, eps):
    m = models("exact", 8, seed=5)
    sh, Wt, _, ptoks = m[:4]
    k_max, depth = 4, 2
    nd, nw, ns = spec_round.uniforms_needed(k_max, depth, trunk)
    u = synth.uniforms(nd + nw + ns, seed=9)
    r = run_round(m, k_max, "topk", depth, 0.0, u[:nd], u[nd:nd + nw], u[nd + nw:], trunk, eps)
    seq = list(ptoks)
    for tok in r.committed:
        lg, _, _ = decoder.prefill(sh, Wt, seq)
        assert tok == int(np.argmax(lg[-1]))
        seq.append(tok)
