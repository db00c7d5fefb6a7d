"""Pins of the oracle's bf16 rounding-point contract (CPU only).

The oracle's bf16 mode is the reference of every bf16 parity test.  Here an
independently written float64 torch forward (its own RMSNorm factoring,
rotary embedding, and attention as one masked softmax over a full key
matrix instead of the oracle's per-row key lists) rounds values through
bfloat16 with torch's own cast at exactly the contract's points:

  attn_in / mlp_in / final_in : each norm's projection input bf16(h g), the
                                row scale 1/rms applied after the product;
  q, k, v                     : q and k after RoPE, v (the cached K and V);
  o                           : the attention output (probabilities not
                                rounded);
  act                         : the SwiGLU product.

The oracle in "bf16_f64" mode (the same rounding points, float64 arithmetic)
must equal it to float64 noise, and must *differ* from it by orders of
magnitude more as soon as any single rounding point is dropped, or an extra
one (the residual stream, the attention probabilities, the scale rounded in
before the product) is added: a missing, extra or misplaced rounding point
in the oracle fails one of these tests.
"""
import numpy as np
import pytest
import torch

from oracle import decoder
from paper_2506_01979_amd import synth
from test_oracle_decoder import GQA

POINTS = ("attn_in", "q", "k", "v", "o", "mlp_in", "act", "final_in")


def bf(x):
    """A float64 tensor stored as bfloat16 from float32 (torch's casts)."""
    return x.to(torch.float32).to(torch.bfloat16).to(torch.float64)


def emulate(shape, W, pk, pv, kv_len, tokens, parents, points=POINTS, extra=()):
    T = lambda a: torch.as_tensor(np.asarray(a, dtype=np.float64))
    rnd = lambda name, x: bf(x) if name in points else x
    N = len(tokens)
    nh, nkv, d = shape.n_heads, shape.n_kv_heads, shape.head_dim
    # ancestors (inclusive) by walking parents; depth = ancestors - 1
    anc = torch.zeros(N, N, dtype=torch.bool)
    for i in range(N):
        j = i
        while j >= 0:
            anc[i, j] = True
            j = int(parents[j])
    pos = kv_len + anc.sum(1).to(torch.float64) - 1
    inv = shape.rope_theta ** (-torch.arange(0, d, 2, dtype=torch.float64) / d)
    ang = pos[:, None] * inv[None, :]
    cos = torch.cat([ang.cos(), ang.cos()], -1)[:, None, :]
    sin = torch.cat([ang.sin(), ang.sin()], -1)[:, None, :]

    def rope(x):
        rot = torch.cat([-x[..., d // 2:], x[..., :d // 2]], -1)
        return x * cos + rot * sin

    # visible keys: every prefix slot, and tree row j for row i iff j is on
    # the path root..i
    allowed = torch.cat([torch.ones(N, kv_len, dtype=torch.bool), anc], 1)

    def norm_proj(name, h, g, mats):
        r = 1.0 / torch.sqrt((h * h).mean(-1, keepdim=True) + shape.rms_eps)
        if "scale_first" in extra:
            a = rnd(name, h * r * T(g))
            return [a @ T(w).T for w in mats]
        a = rnd(name, h * T(g))
        return [(a @ T(w).T) * r for w in mats]

    h = T(W["embed"])[torch.as_tensor(np.asarray(tokens, np.int64))]
    ks, vs = [], []
    for li in range(shape.n_layers):
        L = W["layers"][li]
        q, k, v = norm_proj("attn_in", h, L["attn_norm"], (L["wq"], L["wk"], L["wv"]))
        q = rnd("q", rope(q.view(N, nh, d)))
        k = rnd("k", rope(k.view(N, nkv, d)))
        v = rnd("v", v.view(N, nkv, d))
        ks.append(k.permute(1, 0, 2))
        vs.append(v.permute(1, 0, 2))
        Kall = torch.cat([T(pk[li])[:, :kv_len], k.permute(1, 0, 2)], 1)  # [nkv][keys][d]
        Vall = torch.cat([T(pv[li])[:, :kv_len], v.permute(1, 0, 2)], 1)
        Kh = Kall.repeat_interleave(nh // nkv, 0)
        Vh = Vall.repeat_interleave(nh // nkv, 0)
        s = torch.matmul(q.permute(1, 0, 2), Kh.transpose(1, 2)) / np.sqrt(d)  # [nh][N][keys]
        s = s.masked_fill(~allowed[None], float("-inf"))
        p = torch.softmax(s, -1)
        if "probs" in extra:
            p = bf(p)
        o = rnd("o", torch.matmul(p, Vh).permute(1, 0, 2).reshape(N, nh * d))
        h = h + o @ T(L["wo"]).T
        if "resid" in extra:
            h = bf(h)
        gt, up = norm_proj("mlp_in", h, L["mlp_norm"], (L["wg"], L["wu"]))
        act = rnd("act", gt / (1 + torch.exp(-gt)) * up)
        h = h + act @ T(L["wd"]).T
        if "resid" in extra:
            h = bf(h)
    (logits,) = norm_proj("final_in", h, W["final_norm"], (W["lm_head"],))
    return logits.numpy(), torch.stack(ks).numpy(), torch.stack(vs).numpy()


def relerr(a, b):
    return float(np.max(np.abs(a - b)) / max(1e-300, np.max(np.abs(b))))


def _case(shape, n_prefix, B, k, seed):
    W = synth.model_weights(shape)
    g = np.random.default_rng(seed)
    pk = decoder.round_bf16(g.standard_normal((shape.n_layers, shape.n_kv_heads, n_prefix,
                                               shape.head_dim)).astype(np.float32))
    pv = decoder.round_bf16(g.standard_normal(pk.shape).astype(np.float32))
    parents = synth.branch_parents(B, k)
    toks = g.integers(0, shape.vocab, len(parents))
    return W, pk, pv, toks, parents


SHAPES = {
    "tiny": (synth.SHAPES["tiny"], 16, 2, 4),
    "gqa": (GQA, 9, 3, 2),
    "ragged": (synth.SHAPES["ragged_bf16"], 13, 2, 3),
}


@pytest.fixture(scope="module", params=sorted(SHAPES))
def case(request):
    shape, P, B, k = SHAPES[request.param]
    W, pk, pv, toks, parents = _case(shape, P, B, k, 5)
    ref = decoder.tree_forward(shape, W, pk, pv, P, toks, parents, "bf16_f64")
    return shape, W, pk, pv, P, toks, parents, ref


def test_oracle_bf16_equals_independent_emulation(case):
    shape, W, pk, pv, P, toks, parents, ref = case
    lo, kt, vt = emulate(shape, W, pk, pv, P, toks, parents)
    assert relerr(ref[0], lo) < 1e-10
    assert relerr(ref[1], kt) < 1e-10
    assert relerr(ref[2], vt) < 1e-10


@pytest.mark.parametrize("point", POINTS)
def test_dropping_any_rounding_point_is_detected(case, point):
    shape, W, pk, pv, P, toks, parents, ref = case
    lo, _, _ = emulate(shape, W, pk, pv, P, toks, parents,
                       points=tuple(p for p in POINTS if p != point))
    assert relerr(ref[0], lo) > 1e-6


@pytest.mark.parametrize("extra", ["resid", "probs", "scale_first"])
def test_an_extra_or_moved_rounding_point_is_detected(case, extra):
    shape, W, pk, pv, P, toks, parents, ref = case
    lo, _, _ = emulate(shape, W, pk, pv, P, toks, parents, extra=(extra,))
    assert relerr(ref[0], lo) > 1e-6


def test_float32_bf16_mode_is_the_same_contract():
    """The parity mode ("bf16", float32 arithmetic) runs the same code and
    rounding points as "bf16_f64"; float32 arithmetic moves values across a
    few bf16 rounding boundaries, so the two agree to the bf16 level, well
    inside the 2e-2 parity tolerance, not to float64 noise."""
    shape, P, B, k = SHAPES["tiny"]
    W, pk, pv, toks, parents = _case(shape, P, B, k, 6)
    a = decoder.tree_forward(shape, W, pk, pv, P, toks, parents, "bf16")[0]
    b = decoder.tree_forward(shape, W, pk, pv, P, toks, parents, "bf16_f64")[0]
    assert 0 < relerr(a, b) < 5e-3
