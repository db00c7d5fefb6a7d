"""Pins of the H-RAD predictor oracle (Section "H-RAD", equations for z_t
and s_t): the hidden states it reads against the library Llama model, the
MLP against torch.nn, and the class rule (argmax, lowest index on ties)."""
import numpy as np
import pytest
import torch

from oracle import decoder, hrad
from paper_2506_01979_amd import synth
from test_oracle_decoder import GQA, hf_model, relerr


def _chain_hidden(shape, W, toks):
    hidden = []
    par = synth.chain_parents(len(toks))
    empty = np.zeros((shape.n_layers, shape.n_kv_heads, 0, shape.head_dim))
    lg, _, _ = decoder.tree_forward(shape, W, empty, empty, 0, toks, par, "f64", hidden=hidden)
    return lg, hidden


def test_hidden_states_match_library_model():
    """h^l (residual after layer l) equals the library model's hidden state
    after that layer; the last one, normalised, equals its final output."""
    shape = GQA
    W = synth.model_weights(shape)
    toks = synth.prefix_tokens(shape.vocab, 12)
    _, hidden = _chain_hidden(shape, W, toks)
    assert len(hidden) == shape.n_layers
    m = hf_model(shape, W, exact_rope=True)
    with torch.no_grad():
        out = m(torch.tensor(np.asarray(toks, dtype=np.int64))[None], output_hidden_states=True)
    hs = [h[0].double().numpy() for h in out.hidden_states]
    for l in range(shape.n_layers - 1):
        assert relerr(hidden[l], hs[l + 1]) < 1e-6
    fin = decoder.rms_norm(hidden[-1], W["final_norm"], shape.rms_eps, np.float64)
    assert relerr(fin, hs[-1]) < 1e-6


@pytest.mark.parametrize("K", [1, 2])
def test_tapped_states_are_the_library_models_last_hidden_states(K):
    """The K states H-RAD reads equal the library model's last K reported
    hidden states, whose last entry is the final norm's output."""
    shape = GQA
    W = synth.model_weights(shape)
    toks = synth.prefix_tokens(shape.vocab, 10)
    _, hidden = _chain_hidden(shape, W, toks)
    m = hf_model(shape, W, exact_rope=True)
    with torch.no_grad():
        out = m(torch.tensor(np.asarray(toks, dtype=np.int64))[None], output_hidden_states=True)
    hs = [h[0].double().numpy() for h in out.hidden_states]
    got = hrad.tapped_states(hidden, W["final_norm"], shape.rms_eps, K)
    assert len(got) == K
    for kk in range(K):
        assert relerr(got[kk], hs[len(hs) - K + kk]) < 1e-6


def test_last_hidden_state_gives_the_logits():
    shape = synth.SHAPES["exact"]
    W = synth.model_weights(shape)
    toks = synth.prefix_tokens(shape.vocab, 9)
    lg, hidden = _chain_hidden(shape, W, toks)
    fin = decoder.rms_norm(hidden[-1], W["final_norm"], shape.rms_eps, np.float64)
    assert np.allclose(fin @ np.asarray(W["lm_head"], np.float64).T, lg, rtol=0, atol=1e-12)


def _rand_mlp(din, seed):
    g = np.random.default_rng(seed)
    h1, h2 = hrad.HIDDEN
    return (g.standard_normal((h1, din)) / np.sqrt(din), g.standard_normal(h1) * 0.1,
            g.standard_normal((h2, h1)) / 16.0, g.standard_normal(h2) * 0.1,
            g.standard_normal((hrad.CLASSES, h2)) / 8.0, g.standard_normal(hrad.CLASSES) * 0.1)


def test_mlp_matches_torch():
    din = 5 * 48
    w = _rand_mlp(din, 3)
    z = np.random.default_rng(4).standard_normal(din)
    net = torch.nn.Sequential(torch.nn.Linear(din, 256), torch.nn.ReLU(), torch.nn.Linear(256, 64),
                              torch.nn.ReLU(), torch.nn.Linear(64, 3)).double()
    with torch.no_grad():
        for layer, (wt, bt) in zip((net[0], net[2], net[4]), ((w[0], w[1]), (w[2], w[3]), (w[4], w[5]))):
            layer.weight.copy_(torch.tensor(wt))
            layer.bias.copy_(torch.tensor(bt))
        want = net(torch.tensor(z)).numpy()
    got = hrad.mlp_logits(z, *w)
    assert np.allclose(got, want, rtol=0, atol=1e-12)
    lg, s = hrad.predict(z, *w)
    assert s == int(torch.softmax(torch.tensor(want), 0).argmax())


@pytest.mark.parametrize("b3,want", [([1.0, 5.0, 5.0], 1), ([7.0, 7.0, 7.0], 0), ([0.0, 0.0, 2.0], 2)])
def test_class_is_lowest_index_of_the_largest_logit(b3, want):
    din = 8
    w = list(_rand_mlp(din, 5))
    w[4] = np.zeros((3, 64))
    w[5] = np.asarray(b3)
    lg, s = hrad.predict(np.ones(din), *w)
    assert list(lg) == b3 and s == want


def test_feature_layout():
    a, b, e = np.arange(4.0), np.arange(4.0) + 10, np.arange(4.0) + 100
    z = hrad.features([a, b], e)
    assert list(z) == list(a) + list(b) + list(e)
