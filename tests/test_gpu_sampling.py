"""GPU parity of the softmax statistics, Algorithm 1 and the accept/resample
walk against the oracle, on shared seeded logits (called through the C ABI).

Decisions (accepted rows, branch, emitted token, flags) must be bit-exact
given the same uniforms, except where the oracle's own path passes within
1e-6 of a threshold (|u - p~/q| or |u*W - C_v| / W), where summation order
and exp ulps may legitimately flip a decision.
"""
import json
import os

import numpy as np
import pytest
import torch

from gpu_util import decision_margin, say
from oracle import sampling, tree
from paper_2506_01979_amd import synth

pytestmark = pytest.mark.gpu

TIE = 1e-6


@pytest.fixture(scope="module")
def api():
    from paper_2506_01979_amd import api as A
    assert torch.cuda.is_available()
    return A


def dev(x, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(x))
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


@pytest.mark.parametrize("vocab", [16, 1000, 32000, 128256])
@pytest.mark.parametrize("T", [1.0, 0.7, 0.0])
def test_softmax_stats(api, vocab, T):
    say(f"stats vocab={vocab} T={T}")
    n = 5
    lg = synth.random_logits(n, vocab, 3.0, seed=vocab)
    lg[1, 7] = lg[1].max() + 1.0          # a clear max
    lg[2, [3, 9]] = lg[2].max() + 0.5     # a tie: lowest index wins
    st = api.new_stats(n)
    api.sb_softmax_stats(dev(lg), T, st)
    torch.cuda.synchronize()
    got = api.decode_stats(st)
    for i in range(n):
        ref = sampling.row_stats(lg[i], T)
        assert got["argmax"][i] == ref.argmax
        assert np.float32(got["zmax"][i]) == np.float32(ref.zmax)
        assert abs(got["total"][i] - ref.total) <= 1e-6 * ref.total


def test_softmax_stats_nonfinite(api):
    lg = synth.random_logits(3, 100, 1.0)
    lg[0, 5] = np.nan
    lg[1, 6] = np.inf
    lg[2, 7] = -np.inf      # a masked token is not an error
    st = api.new_stats(3)
    api.sb_softmax_stats(dev(lg), 1.0, st)
    got = api.decode_stats(st)
    assert np.isnan(got["total"][0]) and np.isnan(got["total"][1])
    assert np.isfinite(got["total"][2])


def _golden():
    p = os.path.join(os.path.dirname(__file__), "golden", "accept_cases.txt")
    with open(p) as f:
        return [json.loads(l) for l in f if l.strip() and not l.startswith("#")]


@pytest.mark.parametrize("case", _golden(), ids=lambda c: c["name"])
def test_select_golden(api, case):
    say(f"select golden {case['name']}")
    p = np.asarray(case["p"], dtype=np.float64)
    lg = np.where(p > 0, np.log(np.maximum(p, 1e-300)), -1e30).astype(np.float32)
    V = len(p)
    st = api.new_stats(1)
    api.sb_softmax_stats(dev(lg[None]), 1.0, st)
    q = np.asarray(case["q"], dtype=np.float32)
    out = torch.zeros(3, dtype=torch.int32, device="cuda")
    ws = torch.empty(api.sb_sample_workspace_bytes(V), dtype=torch.uint8, device="cuda")
    api.sb_select_branch(dev(lg), st, 1.0, dev(np.asarray(case["x"], np.int32)), dev(q),
                         dev(np.asarray(case["u"], np.float32)), out, ws)
    o = out.cpu().numpy()
    assert int(o[0]) == case["accepted"]
    assert int(o[1]) == case["token"]


@pytest.mark.parametrize("vocab,n_cand,T", [(1000, 1, 1.0), (1000, 3, 1.0), (32000, 4, 1.0),
                                            (32000, 6, 0.8), (32000, 3, 0.0), (128256, 4, 1.0)])
def test_select_random(api, vocab, n_cand, T):
    say(f"select random vocab={vocab} n_cand={n_cand} T={T}")
    ws = torch.empty(api.sb_sample_workspace_bytes(vocab), dtype=torch.uint8, device="cuda")
    out = torch.zeros(3, dtype=torch.int32, device="cuda")
    checked = 0
    for seed in range(12):
        lg = synth.random_logits(1, vocab, 2.0, seed=100 + seed)[0]
        pst = sampling.row_stats(lg, T)
        p = sampling.target_probs(lg, T, pst)
        qr = synth.softmax_rows(synth.random_logits(1, vocab, 2.0, seed=200 + seed))[0]
        # q partly aligned with p so that acceptances and rejections both occur
        qa = (0.5 * p + 0.5 * qr).astype(np.float32)
        q = np.stack([qa] * n_cand)
        g = np.random.default_rng(seed)
        toks = np.array([g.choice(vocab, p=qa / qa.sum()) for _ in range(n_cand)], np.int32)
        u = synth.uniforms(n_cand + 1, seed=300 + seed)
        tr = []
        res = sampling.branch_select(p, toks, q, u[:n_cand], trace=tr)
        if res.accepted is None:
            y = sampling.draw(res.p_tilde, float(u[n_cand]), tr, n_cand)
            want = (-1, y, res.flags)
        else:
            want = (res.accepted, int(toks[res.accepted]), res.flags)
        st = api.new_stats(1)
        api.sb_softmax_stats(dev(lg[None]), T, st)
        api.sb_select_branch(dev(lg), st, T, dev(toks), dev(q), dev(u), out, ws)
        got = tuple(int(x) for x in out.cpu().numpy())
        if decision_margin(tr, u) < TIE:
            continue
        assert got == want, (seed, got, want)
        checked += 1
    assert checked >= 10


def _walk_case(vocab, parents, T, alpha, seed):
    """Seeded logits, q rows (alpha * p(parent) + (1 - alpha) * q_rand) and
    draft tokens drawn from q."""
    n = len(parents)
    lg = synth.random_logits(n, vocab, 2.0, seed=seed)
    p = np.stack([sampling.target_probs(lg[i], T) for i in range(n)])
    qr = synth.softmax_rows(synth.random_logits(n, vocab, 2.0, seed=seed + 1))
    q = np.zeros((n, vocab), dtype=np.float32)
    g = np.random.default_rng(seed)
    toks = np.zeros(n, dtype=np.int32)
    toks[0] = g.integers(0, vocab)
    for i in range(1, n):
        row = (alpha * p[parents[i]] + (1 - alpha) * qr[i]).astype(np.float32)
        q[i] = row
        toks[i] = g.choice(vocab, p=row.astype(np.float64) / row.astype(np.float64).sum())
    u = synth.uniforms(n, seed=seed + 2)
    return lg, q, toks, u


def _random_tree(n, seed):
    g = np.random.default_rng(seed)
    par = [-1] + [int(g.integers(0, i)) for i in range(1, n)]
    return np.asarray(par, dtype=np.int32)


TREES = [
    ("b4k8", synth.branch_parents(4, 8)),
    ("b1k4", synth.branch_parents(1, 4)),
    ("b8k16", synth.branch_parents(8, 16)),
    ("b2k1", synth.branch_parents(2, 1)),
    ("chain20", synth.chain_parents(20)),
    ("fork4x4x7", synth.fork_parents(4, 4, 7)),
    ("fork6x5x1", synth.fork_parents(6, 5, 1)),
    ("random60", _random_tree(60, 3)),
    ("root_only", np.array([-1], dtype=np.int32)),
    # SB_MAX_ROWS = 256 rows: 15 branches of 17, and a random tree
    ("b15k17", synth.branch_parents(15, 17)),
    ("random256", _random_tree(256, 7)),
]


@pytest.mark.parametrize("name,parents", TREES, ids=[t[0] for t in TREES])
@pytest.mark.parametrize("vocab,T", [(1000, 1.0), (32000, 1.0), (32000, 0.0), (4096, 0.6)])
def test_walk_parity(api, name, parents, vocab, T):
    n = len(parents)
    ws = torch.empty(api.sb_sample_workspace_bytes(vocab), dtype=torch.uint8, device="cuda")
    res_t = api.new_result()
    checked = 0
    outcomes = set()
    cases = 8
    for k in range(cases):
        alpha = (0.2, 0.6, 0.9, 0.99)[k % 4]
        seed = 1000 * k + n + vocab
        say(f"walk {name} vocab={vocab} T={T} case={k} seed={seed}")
        lg, q, toks, u = _walk_case(vocab, parents, T, alpha, seed)
        tr = []
        ref = sampling.accept_resample(toks, parents, lg, T, q, u, trace=tr)
        st = api.new_stats(n)
        dl = dev(lg)
        api.sb_softmax_stats(dl, T, st)
        api.sb_accept_resample(dev(toks), parents, dl, st, T, dev(q), dev(u), res_t, ws)
        got = api.decode_result(res_t)
        if decision_margin(tr, u) < TIE:
            continue
        assert got["path"] == ref.path, (k, got, ref)
        assert got["n_accepted"] == ref.n_accepted
        assert got["branch"] == ref.branch
        assert got["next_token"] == ref.next_token
        assert got["flags"] == ref.flags
        assert got["n_rejected"] == ref.n_rejected
        assert bool(got["bonus"]) == ref.bonus
        outcomes.add((ref.n_accepted, ref.bonus))
        checked += 1
    assert checked >= cases - 2


def test_walk_flags(api):
    vocab = 64
    parents = synth.branch_parents(2, 2)
    lg, q, toks, u = _walk_case(vocab, parents, 1.0, 0.5, 77)
    q[1, toks[1]] = 0.0   # a drafted token with q(x) = 0
    lg[3, 5] = np.nan      # a non-finite target row
    ref = sampling.accept_resample(toks, parents, lg, 1.0, q, u)
    st = api.new_stats(len(parents))
    ws = torch.empty(api.sb_sample_workspace_bytes(vocab), dtype=torch.uint8, device="cuda")
    res_t = api.new_result()
    dl = dev(lg)
    api.sb_softmax_stats(dl, 1.0, st)
    api.sb_accept_resample(dev(toks), parents, dl, st, 1.0, dev(q), dev(u), res_t, ws)
    got = api.decode_result(res_t)
    assert got["flags"] & api.SB_FLAG_NONFINITE
    assert ref.flags & sampling.FLAG_NONFINITE
    assert (got["flags"] & api.SB_FLAG_QZERO) == (ref.flags & sampling.FLAG_QZERO)


def test_host_rejects_bad_tree(api):
    vocab = 32
    ws = torch.empty(api.sb_sample_workspace_bytes(vocab), dtype=torch.uint8, device="cuda")
    lg = torch.zeros((3, vocab), device="cuda")
    st = api.new_stats(3)
    with pytest.raises(api.SBError) as e:
        api.sb_accept_resample(torch.zeros(3, dtype=torch.int32, device="cuda"), [-1, 0, 2], lg,
                               st, 1.0, torch.zeros((3, vocab), device="cuda"),
                               torch.zeros(3, device="cuda"), api.new_result(), ws)
    assert e.value.code == 2
