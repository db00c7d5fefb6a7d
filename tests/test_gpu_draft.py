"""GPU parity of the draft side of a round (Section "Branch Resampling")
against the oracle, through the C ABI.

sb_draft_sample: on the same synthetic logits, each q row within 5e-7
relative of the oracle's (both take float32 exp of the same float32 z and
divide by a float64 total; the two exp implementations and summation
orders differ by a few float32 ulps), T = 0 rows exactly one-hot, and each
token bit-exact unless its uniform lies within 1e-6 (relative to the total)
of a boundary of the oracle's running sum.

sb_draft_round on float32 draft models (float32 GEMMs over K <= 688 put
the logits about 1e-6 from the float64 oracle's): the branch count, the
tree and the tokens bit-exact, the q rows within 2e-5 relative, up to the
first decision the oracle takes within 2e-5 of its threshold (a draw's
uniform against a running sum, B's floor(k_max (1 - q(x_b))) against an
integer, a greedy argmax against the runner-up), where the comparison
stops; the seeds are ones whose rounds have few such ties.  The 68M draft shape in bfloat16
(2 layers, hidden 768, 12 heads of 64, FFN 3072, vocabulary 32000) is
checked by the properties every round has, since its logits carry the
bfloat16 bound.
"""
import numpy as np
import pytest
import torch

from gpu_util import say
from oracle import branching, decoder, drafting
from paper_2506_01979_amd import synth

pytestmark = pytest.mark.gpu

_W = {}
_M = {}


@pytest.fixture(scope="module")
def api():
    from paper_2506_01979_amd import api as A
    assert torch.cuda.is_available()
    return A


def weights(shape):
    if shape.name not in _W:
        _W[shape.name] = synth.model_weights(shape)
    return _W[shape.name]


def model(api, shape):
    if shape.name not in _M:
        _M[shape.name] = api.Model(shape, api.dict_tensors(weights(shape)))
    return _M[shape.name]


def cum_margin(q_row, u):
    C = np.cumsum(np.asarray(q_row, dtype=np.float64))
    W = C[-1]
    return float(np.min(np.abs(C - np.float64(u) * W))) / W if W > 0 else np.inf


@pytest.mark.parametrize("V,T,n", [(32000, 0.7, 6), (32000, 1.0, 16), (1003, 1.3, 5), (16, 0.9, 9),
                                   (32000, 0.0, 4), (128256, 0.8, 3), (1000, 1.0, 64), (1, 1.0, 2),
                                   (2052, 0.9, 3)])
def test_draft_sample_matches_oracle(api, V, T, n):
    seed = V % 97 + n
    logits = synth.random_logits(n + 2, V, scale=3.0, seed=seed)
    g = np.random.default_rng(seed)
    src = g.permutation(n + 2)[:n].astype(np.int32)
    n_out = n + 3
    dst = g.permutation(n_out)[:n].astype(np.int32)
    u = synth.uniforms(n, seed=seed)
    dev = "cuda"
    ld = torch.from_numpy(logits).to(dev)
    stats = api.new_stats(n + 2)
    api.sb_softmax_stats(ld, T, stats)
    toks = torch.full((n_out,), -5, dtype=torch.int32, device=dev)
    q = torch.full((n_out, V), 7.0, dtype=torch.float32, device=dev)
    say(f"draft sample V={V} T={T} n={n}")
    ws = torch.empty(api.sb_draft_sample_workspace_bytes(V, n), dtype=torch.uint8, device=dev)
    api.sb_draft_sample(ld, stats, src, T, torch.from_numpy(u).to(dev), toks, q, dst, ws)
    torch.cuda.synchronize()
    toks, q = toks.cpu().numpy(), q.cpu().numpy()
    for i in range(n):
        qo, to = drafting.sample(logits[src[i]], T, u[i])
        if T > 0:
            np.testing.assert_allclose(q[dst[i]], qo, rtol=5e-7, atol=0)
        else:
            assert np.array_equal(q[dst[i]], qo)
        if T == 0 or cum_margin(qo, u[i]) >= 1e-6:
            assert toks[dst[i]] == to, (i, toks[dst[i]], to)
    rest = np.setdiff1d(np.arange(n_out), dst)
    assert np.all(toks[rest] == -5) and np.all(q[rest] == 7.0)


def gpu_round(api, shape, K, V, P, root, k_max, mode, depth, T, u, trunk=1, eps=float("inf")):
    m = model(api, shape)
    R = trunk + k_max * depth
    k, v = m.new_kv(P + R)
    if P:
        m.load_kv(k, v, K, V, P)
    toks = torch.full((R,), -5, dtype=torch.int32, device="cuda")
    toks[0] = int(root)
    q = torch.full((R, shape.vocab), 7.0, dtype=torch.float32, device="cuda")
    ws = m.draft_round_workspace(k_max, depth, P, trunk)
    B, par, c = m.sb_draft_round(k, v, P, k_max, mode, depth, T, torch.from_numpy(u).cuda(), toks,
                                 q, ws, trunk_max=trunk, confidence=eps)
    torch.cuda.synchronize()
    return B, par, c, toks.cpu().numpy(), q.cpu().numpy()


def first_tie(shape, W, K, V, P, ref, k_max, mode, depth, T, u, trunk=1, eps=float("inf"),
              thr=2e-5):
    """(rows, whole): the oracle's rows before its first decision within thr
    of its threshold, and whether the branch point (B, the tree) is past
    every such decision.  Decisions in the oracle's order: the chain's draws
    and confidence tests, x_b's draw, B's floor(k_max (1 - q(x_b))) against
    an integer, the candidates' draws (or top-k order), the continuations'
    draws; at T = 0 each argmax against the runner-up."""
    lg, _, _ = decoder.tree_forward(shape, W, K, V, P, ref.tokens, ref.parents, "f64")
    B, c = ref.branches, ref.chain
    n = len(ref.tokens)
    if T == 0:
        for r in range(n):
            s = np.sort(lg[r].astype(np.float64))
            if s[-1] - s[-2] < thr * max(1.0, abs(s[-1])):
                kids = [j for j in range(n) if ref.parents[j] == r]
                return (min(kids) if kids else n), r >= c + 1
        return n, True
    for t in range(1, c + 2):                   # chain drafts, then x_b
        row = ref.q[t] if t <= c else ref.q[0]
        tok = ref.tokens[t] if t <= c else ref.x_b
        if cum_margin(row, u[t - 1]) < thr:
            return t, False
        if t < trunk and abs(float(row[tok]) - float(np.float32(eps))) < thr * float(np.float32(eps)):
            return t, False
    x = k_max * (1.0 - float(ref.q[0][ref.x_b]))
    if abs(x - round(x)) < thr * k_max:
        return c + 1, False
    if mode != "topk":
        rem = ref.q[0].astype(np.float64).copy()
        for i in range(B):
            if cum_margin(rem, u[trunk + i]) < thr:
                return c + 1 + i, True
            if mode == "wor":
                rem[ref.tokens[c + 1 + i]] = 0.0
    elif B > 1:
        srt = np.sort(ref.q[0])[::-1]
        if np.min(np.abs(np.diff(srt[:B + 1]))) < thr * srt[0]:
            return c + 1, True
    for d in range(2, depth + 1):
        for i in range(B):
            r = c + 1 + (d - 1) * B + i
            if cum_margin(ref.q[r], u[trunk + k_max * (d - 1) + i]) < thr:
                return r, True
    return n, True


ROUND_CASES = [
    # shape, prefix, k_max, depth, T, seed, trunk_max, confidence
    ("exact", 8, 6, 4, 0.9, 1, 1, None),
    ("exact", 8, 16, 3, 1.0, 2, 1, None),
    ("tiny", 96, 6, 4, 0.8, 7, 1, None),
    ("tiny", 40, 4, 8, 1.2, 7, 1, None),
    ("tiny", 96, 6, 4, 0.8, 5, 1, None),
    ("exact", 8, 6, 5, 0.0, 5, 1, None),
    ("exact", 8, 6, 1, 0.9, 6, 1, None),      # depth 1: the candidates alone
    ("exact", 8, 1, 6, 0.9, 7, 1, None),      # k_max 1: one branch, a chain
    ("exact", 8, 16, 15, 1.0, 8, 1, None),    # 211 rows, near the 256-row limit
    ("exact", 8, 4, 3, 0.9, 28, 6, 0.07),     # a confident chain of 3, then the fork
    ("exact", 8, 4, 3, 0.9, 21, 6, 0.07),     # a chain of 2
    ("exact", 8, 4, 3, 0.9, 8, 6, 0.07),      # a chain of 1
    ("exact", 8, 4, 3, 0.9, 9, 4, 0.0),       # never below 0: the fork after trunk_max - 1
    ("exact", 8, 4, 3, 0.0, 5, 3, 0.5),       # greedy: q(x) = 1, a chain to the end
]


@pytest.mark.parametrize("mode", branching.MODES)
@pytest.mark.parametrize("name,P,k_max,depth,T,seed,trunk,conf", ROUND_CASES)
def test_draft_round_matches_oracle(api, mode, name, P, k_max, depth, T, seed, trunk, conf):
    shape = synth.SHAPES[name]
    W = weights(shape)
    eps = float("inf") if conf is None else conf
    ptoks = synth.prefix_tokens(shape.vocab, P + 1, seed=seed)
    _, K, V = decoder.prefill(shape, W, ptoks[:-1], "f64")
    u = synth.uniforms(drafting.uniforms_needed(k_max, depth, trunk), seed=seed)
    ref = drafting.draft_round(shape, W, K, V, P, int(ptoks[-1]), k_max, mode, depth, T, u,
                               trunk_max=trunk, epsilon=eps)
    say(f"draft round {name} P={P} k_max={k_max} depth={depth} T={T} {mode} trunk={trunk}")
    B, par, c, toks, q = gpu_round(api, shape, K, V, P, ptoks[-1], k_max, mode, depth, T, u,
                                   trunk, eps)
    stop, whole = first_tie(shape, W, K, V, P, ref, k_max, mode, depth, T, u, trunk, eps)
    n = min(stop, len(ref.tokens))
    lo = 0 if whole else 1                     # row 0 is the branch position's row
    assert toks[1:n].tolist() == ref.tokens[1:n].tolist()
    np.testing.assert_allclose(q[lo:n], ref.q[lo:n], rtol=2e-5, atol=1e-12)
    if not whole:
        return
    assert (B, c) == (ref.branches, ref.chain)
    assert par.tolist() == ref.parents.tolist()
    if n == len(ref.tokens):
        assert np.all(q[n:] == 7.0)


def test_draft_round_properties_68m_bf16(api):
    shape = synth.SHAPES["draft68m"]
    P, k_max, depth, T = 256, 6, 5, 1.0
    m = api.Model(shape, api.synth_tensors(shape, seed=7))
    R = 1 + k_max * depth
    k, v = m.new_kv(P + R)
    Kp = np.stack([synth.synthetic_kv(shape, li, P, P, 0, as_bits=True)
                   for li in range(shape.n_layers)])
    Vp = np.stack([synth.synthetic_kv(shape, li, P, P, 1, as_bits=True)
                   for li in range(shape.n_layers)])
    m.load_kv(k, v, Kp, Vp, P)
    for mode in branching.MODES:
        u = synth.uniforms(R, seed=11)
        toks = torch.full((R,), -5, dtype=torch.int32, device="cuda")
        toks[0] = 17
        q = torch.full((R, shape.vocab), 7.0, dtype=torch.float32, device="cuda")
        ws = m.draft_round_workspace(k_max, depth, P)
        say(f"draft round 68m bf16 {mode}")
        B, par, _ = m.sb_draft_round(k, v, P, k_max, mode, depth, T, torch.from_numpy(u).cuda(),
                                     toks, q, ws)
        torch.cuda.synchronize()
        tk, qq = toks.cpu().numpy(), q.cpu().numpy().astype(np.float64)
        assert 1 <= B <= k_max
        assert par.tolist() == [-1] + [0] * B + [1 + (d - 2) * B + i for d in range(2, depth + 1)
                                                for i in range(B)]
        n = 1 + B * depth
        assert np.all((tk[1:n] >= 0) & (tk[1:n] < shape.vocab))
        assert np.all(np.abs(qq[:n].sum(axis=1) - 1.0) < 1e-5)
        assert np.all(qq[np.arange(1, n), tk[1:n]] > 0)
        first = tk[1:1 + B]
        assert len(set(first.tolist())) == B or mode == "iid"
        if mode == "topk":
            assert np.array_equal(qq[1:1 + B], np.eye(shape.vocab)[first])
            assert np.min(qq[0][first]) >= np.sort(qq[0])[-B]
        elif mode == "iid":
            assert np.all(qq[1:1 + B] == qq[0])
        else:
            for i in range(B):
                live = np.ones(shape.vocab, bool)
                live[first[:i]] = False
                assert np.all(qq[1 + i][~live] == 0)
                ratio = qq[1 + i][live] / qq[0][live]
                assert np.allclose(ratio, ratio[0], rtol=1e-6)


def test_draft_round_68m_bf16_replays_the_oracle(api):
    """The 68M bf16 draft's round checked against the oracle by replay: the
    oracle's bfloat16 forward of the round's own tree gives every q row the
    GPU drew from to the bf16 logits bound (2e-2 row-relative, compared as
    T log q, which is the logits up to a per-row constant); every decision
    -- each chain and continuation token, x_b and with it B, the candidates
    and their rows -- is the oracle's draw from the GPU's own q rows with the
    same uniforms, exactly.  The replay draws from the very rows the GPU
    drew from, so the two sides differ only in the float64 summation order
    of the running sums (about 1e-13 relative): no decision of these seeds
    lies within 1e-10 of its threshold, which the test checks."""
    from oracle import sampling
    shape = synth.SHAPES["draft68m"]
    P, k_max, depth, T, trunk = 256, 6, 4, 1.0, 3
    W = synth.model_weights(shape, seed=7)
    m = api.Model(shape, api.synth_tensors(shape, seed=7))
    Kb = np.stack([synth.synthetic_kv(shape, li, P, P, 0, as_bits=True) for li in range(shape.n_layers)])
    Vb = np.stack([synth.synthetic_kv(shape, li, P, P, 1, as_bits=True) for li in range(shape.n_layers)])
    Kf, Vf = synth.bits_to_f32(Kb), synth.bits_to_f32(Vb)
    R = trunk + k_max * depth
    for mode in branching.MODES:
        k, v = m.new_kv(P + R)
        m.load_kv(k, v, Kb, Vb, P)
        u = synth.uniforms(R, seed=23)
        toks = torch.full((R,), -5, dtype=torch.int32, device="cuda")
        toks[0] = 17
        q = torch.full((R, shape.vocab), 7.0, dtype=torch.float32, device="cuda")
        ws = m.draft_round_workspace(k_max, depth, P, trunk)
        say(f"draft round 68m bf16 replay {mode}")
        # threshold 0: every draw is confident, the chain holds trunk - 1
        B, par, c = m.sb_draft_round(k, v, P, k_max, mode, depth, T, torch.from_numpy(u).cuda(),
                                     toks, q, ws, trunk_max=trunk, confidence=0.0)
        torch.cuda.synchronize()
        tk, qg = toks.cpu().numpy(), q.cpu().numpy()
        assert c == trunk - 1 and 1 <= B <= k_max
        n = 1 + c + B * depth
        tree_toks = tk[:n].copy()
        # the oracle forward of the round's tree: row i's logits give the
        # distribution of i's children
        lg, _, _ = decoder.tree_forward(shape, W, Kf, Vf, P, tree_toks, par, "bf16")
        src = {0: c}                                   # row 0 holds q at the branch position
        for i in range(1, c + 1):
            src[i] = i - 1                             # chain drafts
        for i in range(c + 1 + B, n):
            src[i] = int(par[i])                       # continuations
        for i, s in src.items():
            ref = lg[s].astype(np.float64) / T
            got = np.log(qg[i].astype(np.float64)) * 1.0
            d = (got - got.mean()) - (ref - ref.mean())
            assert np.max(np.abs(d)) <= 2e-2 * np.max(np.abs(ref - ref.mean())) * 2, (mode, i)

        def draw(row, uu):
            w = qg[row].astype(np.float64)
            assert cum_margin(qg[row], uu) >= 1e-10
            return sampling.draw(w, float(uu))
        for t in range(1, c + 1):                      # the chain
            assert tk[t] == draw(t, u[t - 1])
        x_b = draw(0, u[c])                            # the branch point
        cand, rows = branching.candidates(qg[0], x_b, k_max, mode, u[trunk:trunk + k_max])
        assert B == len(cand)
        assert tk[c + 1:c + 1 + B].tolist() == cand.tolist()
        np.testing.assert_allclose(qg[c + 1:c + 1 + B], rows, rtol=1e-6, atol=1e-12)
        for d_ in range(2, depth + 1):                 # the continuations
            for i in range(B):
                r = c + 1 + (d_ - 1) * B + i
                assert tk[r] == draw(r, u[trunk + k_max * (d_ - 1) + i])
