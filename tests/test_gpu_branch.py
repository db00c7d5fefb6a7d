"""GPU parity of the branch-point candidates (Section "Branch Resampling")
against the oracle, through the C ABI.

The count B and the candidate tokens must be bit-exact.  Top-k rows are
one-hot and i.i.d. rows copy q, so both are exact too; a row without
replacement is float32(r_v / Z) with Z a float64 sum whose order differs
between the two sides, so it may differ by one float32 ulp (bound: 2.5e-7
relative).  A draw whose uniform lies within 1e-9 of the total of a boundary
of the oracle's running sum is a rounding tie: the comparison stops there.
Sizes: vocabularies of 37 (one partial chunk), 1003 (no 16-byte rows),
32000 and 128256 (the paper's vocabularies), 70001 (a ragged last level-2
entry); q from softmax(N(0,1)/0.7) as the draft distributions elsewhere,
plus sparse, tied and all-zero rows, and an unaligned q.
"""
import numpy as np
import pytest
import torch

from gpu_util import say
from oracle import branching
from paper_2506_01979_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def api():
    from paper_2506_01979_amd import api as A
    assert torch.cuda.is_available()
    return A


def make_q(kind, vocab, seed):
    g = np.random.default_rng(seed)
    if kind == "softmax":
        return synth.draft_q(2, vocab, 0.7, seed=seed)[1]
    if kind == "sparse":                      # 3 tokens with mass
        q = np.zeros(vocab, dtype=np.float32)
        q[g.choice(vocab, 3, replace=False)] = np.array([0.5, 0.3, 0.2], dtype=np.float32)
        return q
    if kind == "tied":                        # four distinct values, many ties
        q = g.integers(1, 5, vocab).astype(np.float32)
        return (q / q.sum()).astype(np.float32)
    if kind == "peaked":                      # one token holds most of the mass
        q = synth.draft_q(2, vocab, 0.7, seed=seed)[1] * np.float32(0.05)
        q[g.integers(vocab)] += np.float32(0.95)
        return q
    if kind == "zero":
        return np.zeros(vocab, dtype=np.float32)
    raise ValueError(kind)


def draw_margin(q, toks, u, mode):
    """Smallest distance, relative to the mass, between u_i * W and the
    oracle's running sum over the remainder each draw used."""
    m = np.inf
    rem = q.astype(np.float64).copy()
    for i, t in enumerate(toks):
        C = np.cumsum(rem)
        W = C[-1]
        if W > 0:
            m = min(m, float(np.min(np.abs(C - np.float64(u[i]) * W))) / W)
        if mode == "wor":
            rem[t] = 0.0
    return m


def run(api, q, x_b, k_max, mode, u, offset=0):
    V = len(q)
    dev = torch.device("cuda")
    qbuf = torch.zeros(V + offset, dtype=torch.float32, device=dev)
    qbuf[offset:] = torch.from_numpy(q).to(dev)
    qd = qbuf[offset:]
    ud = torch.from_numpy(u).to(dev) if u is not None else None
    count = torch.full((1,), -7, dtype=torch.int32, device=dev)
    toks = torch.full((k_max,), -7, dtype=torch.int32, device=dev)
    rows = torch.full((k_max, V), 7.0, dtype=torch.float32, device=dev)
    ws = torch.empty(api.sb_branch_workspace_bytes(), dtype=torch.uint8, device=dev)
    xb = torch.tensor([x_b], dtype=torch.int32, device=dev)
    api.sb_branch_candidates(qd, xb, k_max, mode, ud, count, toks, rows, ws)
    torch.cuda.synchronize()
    return int(count.item()), toks.cpu().numpy(), rows.cpu().numpy()


CASES = [
    # (q kind, vocab, k_max, seed, unaligned q)
    ("softmax", 32000, 6, 11, 0),
    ("softmax", 32000, 16, 12, 0),
    ("softmax", 128256, 6, 13, 0),
    ("softmax", 70001, 16, 14, 0),
    ("softmax", 1003, 16, 15, 0),
    ("softmax", 37, 16, 16, 0),
    ("softmax", 1024, 6, 17, 1),
    ("sparse", 32000, 16, 18, 0),
    ("tied", 4096, 16, 19, 0),
    ("peaked", 32000, 6, 20, 0),
    ("softmax", 1, 16, 21, 0),                # one token: B = 1, that token
    ("softmax", 2, 16, 22, 0),
    ("softmax", 32768, 16, 23, 0),            # the largest vocabulary kept in LDS
    ("softmax", 32769, 16, 24, 0),            # the smallest one read from memory
]


@pytest.mark.parametrize("mode", branching.MODES)
@pytest.mark.parametrize("kind,vocab,k_max,seed,offset", CASES)
def test_candidates_match_oracle(api, mode, kind, vocab, k_max, seed, offset):
    q = make_q(kind, vocab, seed)
    g = np.random.default_rng(seed + 100)
    nz = np.nonzero(q > 0)[0]
    # x_b: a token the draft could have drawn, with a small or large q
    x_b = int(nz[np.argmin(q[nz])]) if seed % 2 else int(nz[g.integers(len(nz))])
    if kind == "peaked":
        x_b = int(np.argmax(q))                # q(x_b) ~ 0.95: B = 1
    u = synth.uniforms(k_max, seed=seed)
    say(f"branch candidates {mode} {kind} V={vocab} k_max={k_max} x_b={x_b} offset={offset}")
    B, toks, rows = run(api, q, x_b, k_max, mode, None if mode == "topk" else u, offset)
    wt, wr = branching.candidates(q, x_b, k_max, mode, u)
    assert B == len(wt)
    assert np.all(toks[B:] == -1)
    assert np.all(rows[B:] == 7.0)            # rows past B untouched
    n = B
    if mode != "topk" and draw_margin(q, wt, u, mode) < 1e-9:
        # compare up to the first draw at a rounding tie
        n = next(i for i in range(B) if draw_margin(q, wt[:i + 1], u, mode) < 1e-9)
    assert np.array_equal(toks[:n], wt[:n]), (toks[:B], wt)
    if mode == "wor":
        np.testing.assert_allclose(rows[:n], wr[:n], rtol=2.5e-7, atol=0)
        assert len(set(toks[:B].tolist())) == B
    else:
        assert np.array_equal(rows[:n], wr[:n])


@pytest.mark.parametrize("mode", branching.MODES)
def test_all_zero_q_gives_no_candidates(api, mode):
    q = make_q("zero", 4096, 0)
    u = synth.uniforms(6, seed=3)
    say(f"branch candidates {mode} all-zero q")
    B, toks, rows = run(api, q, 5, 6, mode, None if mode == "topk" else u)
    assert B == 0 and np.all(toks == -1) and np.all(rows == 7.0)


def test_branch_count_follows_q_of_x_b(api):
    # B = max(1, floor(k_max (1 - q(x_b)))) across the range of q(x_b)
    V = 4096
    for qx in (0.0, 0.05, 1 / 6, 0.25, 0.5, 0.8333, 0.9, 1.0):
        q = np.full(V, (1.0 - qx) / (V - 1), dtype=np.float32)
        q[9] = np.float32(qx)
        say(f"branch count q(x_b)={qx}")
        B, _, _ = run(api, q, 9, 6, "topk", None)
        assert B == branching.branch_count(q[9], 6, int(np.count_nonzero(q > 0)))
    # a token outside the vocabulary counts as q(x_b) = 0: B = k_max
    q = np.full(V, 1.0 / V, dtype=np.float32)
    for xb in (-1, V):
        say(f"branch count x_b={xb}")
        B, _, _ = run(api, q, xb, 6, "topk", None)
        assert B == 6
