"""Pins of the oracle decoder (CPU only).

* The oracle's causal forward matches Hugging Face ``LlamaForCausalLM`` (an
  independent implementation of the paper's target-model family) run as a
  float64 model on the same weights: logits and the cached K/V.  The
  library computes RMSNorm statistics, the attention softmax and (unless
  overridden here) the rotary angles in float32, so agreement is ~1e-7.
* Invariant (a): in the branch-masked tree forward, every branch's rows equal
  a plain causal forward of prefix + root + that branch, and match the
  library model on that sequence.
* bfloat16 emulation rounds like torch's float->bfloat16 cast.
"""
import numpy as np
import pytest
import torch

from oracle import decoder, tree
from paper_2506_01979_amd import synth

transformers = pytest.importorskip("transformers")


def hf_model(shape, W, exact_rope: bool):
    from transformers import LlamaConfig, LlamaForCausalLM

    cfg = LlamaConfig(
        vocab_size=shape.vocab, hidden_size=shape.hidden, intermediate_size=shape.ffn,
        num_hidden_layers=shape.n_layers, num_attention_heads=shape.n_heads,
        num_key_value_heads=shape.n_kv_heads, head_dim=shape.head_dim,
        rope_theta=shape.rope_theta, rms_norm_eps=shape.rms_eps,
        tie_word_embeddings=False, max_position_embeddings=4096,
        attention_bias=False, mlp_bias=False,
    )
    cfg._attn_implementation = "eager"
    m = LlamaForCausalLM(cfg).double().eval()
    t = lambda a: torch.tensor(np.asarray(a, dtype=np.float64))
    with torch.no_grad():
        m.model.embed_tokens.weight.copy_(t(W["embed"]))
        m.lm_head.weight.copy_(t(W["lm_head"]))
        m.model.norm.weight.copy_(t(W["final_norm"]))
        for l, L in enumerate(m.model.layers):
            w = W["layers"][l]
            L.self_attn.q_proj.weight.copy_(t(w["wq"]))
            L.self_attn.k_proj.weight.copy_(t(w["wk"]))
            L.self_attn.v_proj.weight.copy_(t(w["wv"]))
            L.self_attn.o_proj.weight.copy_(t(w["wo"]))
            L.mlp.gate_proj.weight.copy_(t(w["wg"]))
            L.mlp.up_proj.weight.copy_(t(w["wu"]))
            L.mlp.down_proj.weight.copy_(t(w["wd"]))
            L.input_layernorm.weight.copy_(t(w["attn_norm"]))
            L.post_attention_layernorm.weight.copy_(t(w["mlp_norm"]))
        if exact_rope:
            # the library forces its rotary angles to float32; run the same
            # computation in float64 so the remaining comparison is exact
            rot = m.model.rotary_emb
            d = shape.head_dim
            inv = 1.0 / (shape.rope_theta ** (torch.arange(0, d, 2, dtype=torch.float64) / d))

            def forward64(x, position_ids):
                freqs = position_ids[:, :, None].double() * inv[None, None, :]
                emb = torch.cat((freqs, freqs), dim=-1)
                return emb.cos().to(x.dtype), emb.sin().to(x.dtype)

            rot.forward = forward64
    return m


def hf_forward(m, tokens):
    with torch.no_grad():
        out = m(torch.tensor(np.asarray(tokens, dtype=np.int64))[None], use_cache=True)
    logits = out.logits[0].double().numpy()
    pkv = out.past_key_values
    ks, vs = [], []
    for l in range(len(m.model.layers)):
        if hasattr(pkv, "layers"):
            k, v = pkv.layers[l].keys, pkv.layers[l].values
        else:
            k, v = pkv[l]
        ks.append(k[0].double().numpy())
        vs.append(v[0].double().numpy())
    return logits, np.stack(ks), np.stack(vs)


def relerr(a, b):
    return float(np.max(np.abs(a - b)) / max(1e-30, np.max(np.abs(b))))


GQA = synth.Shape("gqa_test", 2, 128, 4, 2, 32, 344, 48, "f32")


@pytest.mark.parametrize("shape", [synth.SHAPES["exact"], GQA], ids=["exact", "gqa"])
def test_causal_forward_matches_hf_llama(shape):
    W = synth.model_weights(shape)
    toks = synth.prefix_tokens(shape.vocab, 24)
    lo, K, V = decoder.prefill(shape, W, toks, "f64")
    # the library keeps RMSNorm statistics and the attention softmax in
    # float32 even in a float64 model, hence 1e-6 rather than 1e-12
    for exact, tol in ((True, 1e-6), (False, 1e-5)):
        m = hf_model(shape, W, exact_rope=exact)
        lh, Kh, Vh = hf_forward(m, toks)
        assert relerr(lo, lh) < tol
        assert relerr(K, Kh) < tol
        assert relerr(V, Vh) < tol


def test_causal_forward_matches_hf_tiny_shape():
    shape = synth.SHAPES["tiny"]
    W = synth.model_weights(shape)
    toks = synth.prefix_tokens(shape.vocab, 40)
    lo, _, _ = decoder.prefill(shape, W, toks, "f64")
    lh, _, _ = hf_forward(hf_model(shape, W, exact_rope=True), toks)
    assert relerr(lo, lh) < 1e-6


@pytest.mark.parametrize("wname,shape", [("exact", synth.SHAPES["exact"]), ("gqa", GQA)])
def test_branch_mask_equals_per_branch_forward(wname, shape):
    """Invariant (a): branch-masked verification == each branch alone."""
    W = synth.model_weights(shape)
    P = 12
    B, k = 3, 3
    ptoks = synth.prefix_tokens(shape.vocab, P)
    _, Kp, Vp = decoder.prefill(shape, W, ptoks[:-1], "f64")
    parents = synth.branch_parents(B, k)
    g = np.random.default_rng(7)
    toks = g.integers(0, shape.vocab, len(parents)).astype(np.int32)
    toks[0] = ptoks[-1]
    lt, kt, vt = decoder.tree_forward(shape, W, Kp, Vp, P - 1, toks, parents, "f64")
    m = hf_model(shape, W, exact_rope=True)
    for b in range(B):
        rows = [0] + [1 + b * k + j for j in range(k)]
        lc, kc, vc = decoder.tree_forward(shape, W, Kp, Vp, P - 1, toks[rows],
                                          synth.chain_parents(len(rows)), "f64")
        assert np.allclose(lt[rows], lc, rtol=0, atol=1e-12 * np.abs(lc).max())
        assert np.allclose(kt[:, :, rows], kc, rtol=0, atol=1e-12 * np.abs(kc).max())
        assert np.allclose(vt[:, :, rows], vc, rtol=0, atol=1e-12 * np.abs(vc).max())
        # the same rows from the library model on prefix + branch
        lh, _, _ = hf_forward(m, np.concatenate([ptoks, toks[rows[1:]]]))
        assert relerr(lt[rows], lh[P - 1:]) < 1e-6


def test_fork_tree_equals_chain_plus_candidate():
    """The chain-plus-fork shape: every root-to-leaf path of the tree
    forward equals a causal forward of the prefix followed by that path
    (the trunk, one candidate, its continuation), checked against the
    library model."""
    shape = synth.SHAPES["exact"]
    W = synth.model_weights(shape)
    P, trunk, B, d = 10, 3, 3, 2
    par = synth.fork_parents(trunk, B, d)
    assert list(par) == [-1, 0, 1, 2, 3, 4, 3, 6, 3, 8]
    assert tree.children(par, trunk) == [4, 6, 8]
    ptoks = synth.prefix_tokens(shape.vocab, P)
    _, Kp, Vp = decoder.prefill(shape, W, ptoks[:-1], "f64")
    g = np.random.default_rng(11)
    toks = g.integers(0, shape.vocab, len(par)).astype(np.int32)
    toks[0] = ptoks[-1]
    lt, _, _ = decoder.tree_forward(shape, W, Kp, Vp, P - 1, toks, par, "f64")
    m = hf_model(shape, W, exact_rope=True)
    for leaf in (5, 7, 9):
        rows = tree.root_path(par, leaf)
        lh, _, _ = hf_forward(m, np.concatenate([ptoks, toks[rows[1:]]]))
        assert relerr(lt[rows], lh[P - 1:]) < 1e-6


def test_tree_positions_and_paths():
    par = synth.branch_parents(2, 3)
    assert list(par) == [-1, 0, 1, 2, 0, 4, 5]
    assert list(tree.depths(par)) == [0, 1, 2, 3, 1, 2, 3]
    assert tree.root_path(par, 6) == [0, 4, 5, 6]
    assert tree.children(par, 0) == [1, 4]
    with pytest.raises(ValueError):
        tree.validate([-1, 1])
    with pytest.raises(ValueError):
        tree.validate([0, 0])


def test_round_bf16_matches_torch_cast():
    g = np.random.default_rng(3)
    x = np.concatenate([g.standard_normal(100000).astype(np.float32) * 10,
                        np.array([0.0, -0.0, 1e-40, 3.0e38, 1.00390625, 1.01171875], np.float32)])
    want = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    got = decoder.round_bf16(x)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


def test_bf16_mode_close_to_f32():
    shape = synth.SHAPES["small_bf16"]
    W = synth.model_weights(shape)
    toks = synth.prefix_tokens(shape.vocab, 20)
    l32, _, _ = decoder.prefill(shape, W, toks, "f32")
    l16, _, _ = decoder.prefill(shape, W, toks, "bf16")
    assert relerr(l16, l32) < 5e-2
    assert relerr(l16, l32) > 0
