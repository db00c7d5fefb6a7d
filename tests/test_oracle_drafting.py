"""Pins of the draft-side oracle: the draft's sampled rows against the
library softmax and an independent inverse CDF, and a whole drafting round
(Section "Branch Resampling") against the library Llama model run on each
branch's plain token sequence."""
import numpy as np
import pytest
import scipy.special
import torch

from oracle import branching, decoder, drafting
from paper_2506_01979_amd import synth
from test_oracle_decoder import hf_model


@pytest.mark.parametrize("T", [0.7, 1.0, 1.6])
def test_sample_is_the_softmax_row_and_its_inverse_cdf(T):
    g = np.random.default_rng(3)
    for trial in range(20):
        l = (g.standard_normal(700) * 3).astype(np.float32)
        u = np.float32(g.random())
        q, t = drafting.sample(l, T, u)
        # z = fl32(l * fl32(1/T)), as the target's statistics take it.  Against
        # the library softmax of that z: float32 rounding of z - max z (2^-24
        # |z - max z|), of exp and of the stored value (a few 2^-24)
        z = (l * (np.float32(1) / np.float32(T))).astype(np.float64)
        eps = 2.0 ** -24
        assert q.dtype == np.float32
        sm = scipy.special.softmax(z)
        assert np.all(np.abs(q - sm) / sm < 2 * eps * np.abs(z - z.max()) + 8 * eps)
        # against the exact l / T: add z's own rounding, 2^-24 |z| per entry,
        # which enters through the entry and through the normaliser
        ref = scipy.special.softmax(l.astype(np.float64) / np.float64(T))
        bound = 2 * eps * (np.abs(z - z.max()) + np.abs(z) + np.abs(z).max()) + 8 * eps
        assert np.all(np.abs(q - ref) / ref < bound)
        C = np.cumsum(q.astype(np.float64))
        assert t == int(np.searchsorted(C, np.float64(u) * C[-1], side="right"))


def test_sample_greedy_is_one_hot_at_the_lowest_argmax():
    l = np.array([0.5, 2.0, -1.0, 2.0], dtype=np.float32)
    q, t = drafting.sample(l, 0.0, 0.99)
    assert t == 1 and np.array_equal(q, np.array([0, 1, 0, 0], dtype=np.float32))


SHAPE = synth.SHAPES["exact"]


def _round(mode, T, k_max, depth, seed):
    W = synth.model_weights(SHAPE, seed=seed)
    ptoks = synth.prefix_tokens(SHAPE.vocab, 9, seed=seed)
    _, K, V = decoder.prefill(SHAPE, W, ptoks[:-1], "f64")
    u = synth.uniforms(drafting.uniforms_needed(k_max, depth), seed=seed)
    r = drafting.draft_round(SHAPE, W, K, V, len(ptoks) - 1, int(ptoks[-1]), k_max, mode, depth,
                             T, u)
    return W, ptoks, u, r


def _branch_rows(r, i, depth):
    return [0] + [1 + (d - 1) * r.branches + i for d in range(1, depth + 1)]


@pytest.mark.parametrize("mode", branching.MODES)
def test_round_layout_and_branch_point(mode):
    k_max, depth = 6, 4
    W, ptoks, u, r = _round(mode, 0.9, k_max, depth, 4)
    B = r.branches
    assert B == branching.branch_count(r.q[0][r.x_b], k_max, int(np.count_nonzero(r.q[0] > 0)))
    assert len(r.tokens) == len(r.parents) == len(r.q) == 1 + B * depth
    want_par = [-1] + [0] * B + [1 + (d - 2) * B + i for d in range(2, depth + 1) for i in range(B)]
    assert r.parents.tolist() == want_par
    # x_b is the draw from the root's row with u[0]; the first level is the candidate set
    C = np.cumsum(r.q[0].astype(np.float64))
    assert r.x_b == int(np.searchsorted(C, np.float64(u[0]) * C[-1], side="right"))
    ct, cr = branching.candidates(r.q[0], r.x_b, k_max, mode, u[1:1 + k_max])
    assert r.tokens[1:1 + B].tolist() == ct.tolist()
    assert np.array_equal(r.q[1:1 + B], cr)


@pytest.mark.parametrize("mode", branching.MODES)
def test_round_continuations_match_library_model(mode):
    """Each branch's rows at depth >= 2 carry softmax(library logits / T) of
    the branch's own plain sequence (prefix, root, its earlier tokens), and
    each token is the inverse-CDF draw of its row with its uniform."""
    k_max, depth, T = 6, 4, 0.9
    W, ptoks, u, r = _round(mode, T, k_max, depth, 5)
    m = hf_model(SHAPE, W, exact_rope=True)
    B = r.branches
    for i in range(B):
        rows = _branch_rows(r, i, depth)
        seq = np.concatenate([ptoks, r.tokens[rows[1:]]]).astype(np.int64)
        with torch.no_grad():
            lg = m(torch.tensor(seq)[None]).logits[0].double().numpy()
        for d in range(2, depth + 1):
            row = rows[d]
            ref = scipy.special.softmax(lg[len(ptoks) + d - 2] / np.float64(np.float32(T)))
            assert np.max(np.abs(r.q[row] - ref)) < 1e-6
            C = np.cumsum(r.q[row].astype(np.float64))
            uu = u[1 + k_max * (d - 1) + i]
            assert r.tokens[row] == int(np.searchsorted(C, np.float64(uu) * C[-1], side="right"))
        # the root's row: the library's distribution after the prefix
        ref0 = scipy.special.softmax(lg[len(ptoks) - 1] / np.float64(np.float32(T)))
        assert np.max(np.abs(r.q[0] - ref0)) < 1e-6


def test_greedy_round_is_one_branch_of_greedy_decoding():
    # at T = 0 q is one-hot, so B = 1 and the branch is the library's greedy path
    depth = 5
    W, ptoks, u, r = _round("topk", 0.0, 6, depth, 6)
    assert r.branches == 1
    m = hf_model(SHAPE, W, exact_rope=True)
    seq = list(ptoks)
    for _ in range(depth):
        with torch.no_grad():
            lg = m(torch.tensor(np.asarray(seq, dtype=np.int64))[None]).logits[0, -1].numpy()
        seq.append(int(np.argmax(lg)))
    assert r.tokens[1:].tolist() == seq[len(ptoks):]


@pytest.mark.parametrize("mode", branching.MODES)
def test_round_with_a_confident_chain(mode):
    """The branch point is the first drafted token below the confidence
    threshold: the chain before it holds the library model's draws (each
    token at or above the threshold), x_b is below it (or the last allowed),
    and every branch continues after the chain."""
    k_max, depth, T, trunk_max, eps = 4, 3, 0.9, 6, 0.07
    seed = 8
    W = synth.model_weights(SHAPE, seed=seed)
    ptoks = synth.prefix_tokens(SHAPE.vocab, 9, seed=seed)
    _, K, V = decoder.prefill(SHAPE, W, ptoks[:-1], "f64")
    u = synth.uniforms(drafting.uniforms_needed(k_max, depth, trunk_max), seed=seed)
    r = drafting.draft_round(SHAPE, W, K, V, len(ptoks) - 1, int(ptoks[-1]), k_max, mode, depth, T,
                             u, trunk_max=trunk_max, epsilon=eps)
    c, B = r.chain, r.branches
    assert 1 <= c < trunk_max                      # this seed drafts a chain, then branches
    assert len(r.tokens) == 1 + c + B * depth
    assert r.parents.tolist() == ([-1] + list(range(c)) + [c] * B +
                                  [c + 1 + (d - 2) * B + i for d in range(2, depth + 1)
                                   for i in range(B)])
    m = hf_model(SHAPE, W, exact_rope=True)
    chain = r.tokens[1:1 + c]
    with torch.no_grad():
        lg = m(torch.tensor(np.concatenate([ptoks, chain]).astype(np.int64))[None]).logits[0]
    lg = lg.double().numpy()
    for t in range(1, c + 2):                      # chain tokens, then x_b
        ref = scipy.special.softmax(lg[len(ptoks) + t - 2] / np.float64(np.float32(T)))
        row = r.q[t] if t <= c else r.q[0]
        assert np.max(np.abs(row - ref)) < 1e-6
        C = np.cumsum(row.astype(np.float64))
        tok = r.tokens[t] if t <= c else r.x_b
        assert tok == int(np.searchsorted(C, np.float64(u[t - 1]) * C[-1], side="right"))
        assert (row[tok] >= np.float32(eps)) == (t <= c)
    ct, cr = branching.candidates(r.q[0], r.x_b, k_max, mode, u[trunk_max:trunk_max + k_max])
    assert r.tokens[1 + c:1 + c + B].tolist() == ct.tolist()
    for i in range(B):                             # each branch continues after the chain
        rows = [1 + c + (d - 1) * B + i for d in range(1, depth + 1)]
        seq = np.concatenate([ptoks, chain, r.tokens[rows]]).astype(np.int64)
        with torch.no_grad():
            lb = m(torch.tensor(seq)[None]).logits[0].double().numpy()
        for d in range(2, depth + 1):
            ref = scipy.special.softmax(lb[len(ptoks) + c + d - 2] / np.float64(np.float32(T)))
            assert np.max(np.abs(r.q[rows[d - 1]] - ref)) < 1e-6
