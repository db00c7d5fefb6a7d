"""Pins of the branch-point candidate oracle (Section "Branch Resampling";
reading R1: each candidate carries the distribution it was drawn from)."""
import numpy as np
import pytest

from oracle import branching


@pytest.mark.parametrize("q,k,nnz,want", [(0.9, 6, None, 1), (0.25, 6, None, 4), (0.0, 6, None, 6),
                                          (0.5, 6, None, 3), (1.0, 6, None, 1), (0.1, 6, None, 5),
                                          (0.0, 6, 2, 2), (0.4, 16, None, 9)])
def test_branch_count_closed_form(q, k, nnz, want):
    # floor(k_max (1 - q(x_b))), at least 1, at most the tokens with mass;
    # q is the float32 value (0.1 -> 0.100000001: 6 * 0.8999... = 5.39...)
    assert branching.branch_count(q, k, nnz) == want


def _q(V, seed, zeros=0):
    g = np.random.default_rng(seed)
    q = g.random(V).astype(np.float32) ** 3
    if zeros:
        q[g.choice(V, zeros, replace=False)] = 0.0
    return (q / q.sum()).astype(np.float32)


def test_topk_is_the_largest_entries_lowest_index_first():
    q = _q(50, 1)
    q[7] = q[9] = q[30] = np.float32(0.5)    # a three-way tie above every other entry
    toks, rows = branching.candidates(q, 3, 6, "topk", None)
    B = branching.branch_count(q[3], 6, 50)
    want = sorted(range(50), key=lambda v: (-float(q[v]), v))[:B]
    assert list(toks) == want and list(toks[:3]) == [7, 9, 30]
    assert np.array_equal(rows, np.eye(50, dtype=np.float32)[want])


def test_iid_draws_are_inverse_cdf_of_q():
    q = _q(40, 2)
    u = np.random.default_rng(3).random(16).astype(np.float32)
    toks, rows = branching.candidates(q, 0, 16, "iid", u)
    C = np.cumsum(q.astype(np.float64))
    for i, t in enumerate(toks):
        assert t == int(np.searchsorted(C, np.float64(u[i]) * C[-1], side="right"))
        assert np.array_equal(rows[i], q)


def test_without_replacement_rows_are_the_renormalised_remainders():
    q = _q(30, 4, zeros=20)                # 10 tokens with mass: B is capped by them
    u = np.random.default_rng(5).random(16).astype(np.float32)
    toks, rows = branching.candidates(q, 0, 16, "wor", u)
    B = branching.branch_count(q[0], 16, 10)
    assert len(toks) == B and len(set(toks.tolist())) == B
    rem = q.astype(np.float64).copy()
    for i, t in enumerate(toks):
        assert abs(float(rows[i].astype(np.float64).sum()) - 1.0) < 1e-6
        assert np.all(rows[i][toks[:i]] == 0)
        live = rem > 0
        ratio = rows[i][live].astype(np.float64) / rem[live]
        assert np.allclose(ratio, ratio[0], rtol=1e-6)
        C = np.cumsum(rem)
        assert t == int(np.searchsorted(C, np.float64(u[i]) * C[-1], side="right"))
        rem[t] = 0.0


def test_without_replacement_pair_law_by_enumeration():
    # P(first = a, second = b) = q_a q_b / (1 - q_a): enumerate (u0, u1) on a
    # midpoint grid, so each frequency is exact up to the grid spacing
    q = np.array([0.1, 0.4, 0.2, 0.3], dtype=np.float32)
    n = 100
    freq = np.zeros((4, 4))
    for i in range(n):
        for j in range(n):
            u = np.array([(i + 0.5) / n, (j + 0.5) / n], dtype=np.float32)
            toks, _ = branching.candidates(q, 0, 3, "wor", u)   # B = floor(3 * 0.9) = 2
            freq[toks[0], toks[1]] += 1.0 / (n * n)
    qd = q.astype(np.float64)
    want = np.array([[0.0 if a == b else qd[a] * qd[b] / (1 - qd[a]) for b in range(4)]
                     for a in range(4)])
    assert np.abs(freq - want).max() < 2.0 / n


@pytest.mark.parametrize("mode", branching.MODES)
def test_candidates_through_algorithm1_emit_the_target_distribution(mode):
    """R1 end to end: the candidates and the rows they carry, tested by
    Algorithm 1 at the root (sampling.accept_resample over the root and B
    children), emit a first token distributed exactly as p.  Exact
    enumeration over the candidate draws' uniforms and the walk's together."""
    from oracle import sampling
    from walk_enum import enumerate_outcomes
    V = 6
    k = np.array([9, 3, 7, 2, 6, 5], dtype=np.int64)          # dyadic q: draws and rows agree
    q = (k / k.sum()).astype(np.float32)
    q = (np.round(q.astype(np.float64) * 2 ** 20) / 2 ** 20).astype(np.float32)
    q[0] += np.float32(1.0) - q.sum(dtype=np.float32)
    p = np.array([0.05, 0.3, 0.1, 0.25, 0.2, 0.1])
    x_b, k_max = 3, 4                                           # B = floor(4 (1 - q_3)) = 3
    B = branching.branch_count(q[x_b], k_max, V)
    assert B == 3
    logits = np.zeros((1 + B, V), dtype=np.float32)
    logits[0] = np.log(p).astype(np.float32)
    p_used = sampling.target_probs(logits[0], 1.0)
    parents = [-1] + [0] * B

    def run(u):
        tr = []
        toks, rows = branching.candidates(q, x_b, k_max, mode, u[:B], trace=tr)
        qa = np.zeros((1 + B, V), dtype=np.float32)
        qa[1:] = rows
        wt = []
        r = sampling.accept_resample([0] + [int(t) for t in toks], parents, logits, 1.0, qa,
                                     u[B:], trace=wt)
        tr += [(ev[0], ev[1] + B) + tuple(ev[2:]) for ev in wt]
        r.first = int(toks[r.path[1] - 1]) if r.n_accepted else r.next_token
        return r, tr

    def relevant(r, tr):
        # after an accepted child the bonus draw no longer moves the first token
        return len(tr) - 1 if r.n_accepted else len(tr)

    out = enumerate_outcomes(run, 2 * B + 1, lambda r: r.first, relevant)
    dist = np.zeros(V)
    for v, pr in out.items():
        dist[v] += pr
    # rows without replacement are float32 roundings of the remainders the
    # draws use, ~1e-8 apart
    tol = 1e-6 if mode == "wor" else 1e-9
    assert abs(dist.sum() - 1.0) < tol
    assert np.max(np.abs(dist - p_used)) < tol
