"""GPU parity of sb_verify_forward against the oracle decoder.

Logits must match per row within 1e-4 (float32 models, against the float64
oracle) or 2e-2 (bfloat16 models, against the oracle's bfloat16 emulation)
relative to the row's largest logit; the K/V the step writes for the tree
rows must match to the same bound.  Shapes span several GEMM tiles, ragged K
(ffn 688, 600), ragged vocabularies (1000, 1001), a hidden width that is not
a multiple of 16 (328), ragged attention chunks, GQA, both head widths and
5..137-row trees (the O projection applies the post-attention RMSNorm up to
128 rows and hands it to a separate kernel above), the paper's
chain-plus-fork verification shape (a chain of drafts, then B candidates
with or without continuations), and 32 KV heads on a narrow model (few key
ranges per head).  Invariant (a) -- branch-masked rows equal
each branch run alone -- is checked on the GPU path too.
"""
import numpy as np
import pytest
import torch

from gpu_util import row_relerr, say
from oracle import decoder, sampling
from paper_2506_01979_amd import synth

pytestmark = pytest.mark.gpu

_WEIGHTS = {}
_MODELS = {}


@pytest.fixture(scope="module")
def api():
    from paper_2506_01979_amd import api as A
    assert torch.cuda.is_available()
    return A


def weights(shape):
    if shape.name not in _WEIGHTS:
        _WEIGHTS[shape.name] = synth.model_weights(shape)
    return _WEIGHTS[shape.name]


def model(api, shape):
    if shape.name not in _MODELS:
        _MODELS[shape.name] = api.Model(shape, api.dict_tensors(weights(shape)))
    return _MODELS[shape.name]


def tol(shape):
    return 2e-2 if shape.dtype == "bf16" else 1e-4


def mode(shape):
    return "bf16" if shape.dtype == "bf16" else "f64"


def gpu_forward(api, m, Kp, Vp, kv_len, tokens, parents, T=1.0, cap=None, stats_out=None):
    """Logits and cache of one sb_verify_forward call; the row statistics
    are appended to stats_out when given."""
    n = len(parents)
    cap = cap or kv_len + n + 8
    k, v = m.new_kv(cap)
    if kv_len:
        m.load_kv(k, v, Kp, Vp, kv_len)
    logits = torch.empty((n, m.shape.vocab), dtype=torch.float32, device="cuda")
    stats = api.new_stats(n)
    ws = m.workspace(n, kv_len)
    toks = torch.from_numpy(np.asarray(tokens, np.int32)).cuda()
    m.sb_verify_forward(k, v, kv_len, toks, parents, T, logits, stats, ws)
    torch.cuda.synchronize()
    if stats_out is not None:
        stats_out.append(api.decode_stats(stats))
    return logits.cpu().numpy(), k, v


def check_stats(st, logits, T):
    """The forward's row statistics against the oracle's on the same logits:
    zmax and argmax exact, total within 1e-6 relative (NaN where the
    oracle's is NaN)."""
    for i in range(logits.shape[0]):
        rs = sampling.row_stats(logits[i], T)
        assert st["argmax"][i] == rs.argmax, (i, st["argmax"][i], rs.argmax)
        assert np.float32(st["zmax"][i]) == np.float32(rs.zmax), i
        if np.isnan(rs.total):
            assert np.isnan(st["total"][i]), i
        else:
            assert abs(st["total"][i] - rs.total) <= 1e-6 * rs.total, (i, st["total"][i], rs.total)


CASES = [
    # shape, prefix P, tree
    ("tiny", 128, ("branch", 2, 4)),
    ("exact", 8, ("branch", 3, 3)),
    ("tiny", 40, ("chain", 30)),
    ("small_bf16", 128, ("branch", 2, 4)),
    ("small_bf16", 300, ("branch", 4, 8)),
    ("small_gqa_bf16", 300, ("branch", 4, 8)),
    ("small_h128_bf16", 200, ("branch", 8, 16)),
    ("small_bf16", 1, ("chain", 40)),
    ("ragged_bf16", 300, ("branch", 4, 8)),
    ("ragged_bf16", 90, ("branch", 8, 17)),
    ("heads32_bf16", 300, ("branch", 4, 8)),
    ("heads32_bf16", 90, ("branch", 8, 7)),
    ("small_bf16", 300, ("fork", 4, 4, 7)),
    ("tiny", 64, ("fork", 6, 3, 1)),
    # head_dim 128 with every row of a KV head in one block of at most 48
    # rows (the 7B step's attention shape): ranges of 4 steps, 8 ranges, a
    # key count that ends inside a 16-byte V^T chunk, grouped queries
    ("small_h128_bf16", 200, ("branch", 4, 8)),
    ("small_h128_bf16", 1000, ("branch", 2, 4)),
    ("small_h128_bf16", 37, ("chain", 20)),
    ("small_h128_bf16", 2047, ("branch", 4, 8)),
    ("gqa128_bf16", 300, ("branch", 4, 4)),
    ("gqa128_bf16", 1, ("chain", 9)),
    # trees of 65 .. 80 rows (5 token tiles)
    ("small_gqa_bf16", 300, ("branch", 8, 8)),
    ("small_h128_bf16", 100, ("branch", 5, 15)),
    # more than 16 rounds of (KV head, key range, row block) units: each
    # workgroup walks the three row blocks of its key range
    ("heads32_bf16", 11000, ("branch", 8, 16)),
    # long prefixes over many one-step workgroups (head_dim 64 and 128, one
    # and three row blocks, grouped queries, up to 95 key ranges)
    ("heads32_bf16", 3000, ("branch", 8, 16)),
    ("heads32_bf16", 5000, ("branch", 4, 8)),
    ("gqa128_bf16", 24000, ("branch", 8, 16)),
    # trees of 145 .. 192 rows (12 token tiles in the wide GEMMs)
    ("ragged_bf16", 90, ("branch", 10, 17)),
    ("small_h128_bf16", 500, ("branch", 12, 13)),
    # the largest trees (SB_MAX_ROWS = 256 rows): 15 x 17 branches, a
    # 256-row chain (ancestor bit 255)
    ("small_bf16", 64, ("branch", 15, 17)),
    ("small_gqa_bf16", 8, ("chain", 256)),
]


def tree_of(spec):
    if spec[0] == "branch":
        return synth.branch_parents(spec[1], spec[2])
    if spec[0] == "fork":
        return synth.fork_parents(spec[1], spec[2], spec[3])
    return synth.chain_parents(spec[1])


@pytest.mark.parametrize("sname,P,spec", CASES, ids=[f"{c[0]}-P{c[1]}-{c[2]}" for c in CASES])
def test_verify_forward_parity(api, sname, P, spec):
    shape = synth.SHAPES[sname]
    say(f"forward parity {sname} P={P} tree={spec}")
    W = weights(shape)
    parents = tree_of(spec)
    n = len(parents)
    ptoks = synth.prefix_tokens(shape.vocab, P)
    kv_len = P - 1
    if kv_len > 2500:
        # a long prefix: seeded N(0, 1) keys and values stand in for a
        # prefill (the oracle's prefill is quadratic in the prefix)
        gk = np.random.default_rng(P)
        dims = (shape.n_layers, shape.n_kv_heads, kv_len, shape.head_dim)
        Kp, Vp = gk.standard_normal(dims), gk.standard_normal(dims)
        if mode(shape) == "bf16":
            Kp, Vp = decoder.round_bf16(Kp.astype(np.float32)), decoder.round_bf16(Vp.astype(np.float32))
    elif kv_len:
        _, Kp, Vp = decoder.prefill(shape, W, ptoks[:-1], mode(shape))
    else:
        Kp = Vp = np.zeros((shape.n_layers, shape.n_kv_heads, 0, shape.head_dim))
    g = np.random.default_rng(P + n)
    toks = g.integers(0, shape.vocab, n).astype(np.int32)
    toks[0] = ptoks[-1]
    ref, kt, vt = decoder.tree_forward(shape, W, Kp, Vp, kv_len, toks, parents, mode(shape))
    m = model(api, shape)
    st = []
    got, k, v = gpu_forward(api, m, Kp, Vp, kv_len, toks, parents, stats_out=st)
    err = row_relerr(got, ref)
    say(f"  logits row-relative error {err:.3e}")
    assert err < tol(shape)
    check_stats(st[0], got, 1.0)
    kg, vg = m.read_kv(k, v, kv_len, n)
    assert row_relerr(kg.reshape(-1, shape.head_dim), kt.reshape(-1, shape.head_dim)) < tol(shape) * 5
    assert row_relerr(vg.reshape(-1, shape.head_dim), vt.reshape(-1, shape.head_dim)) < tol(shape) * 5
    # the prefix slots are untouched
    if kv_len:
        kp, vp = m.read_kv(k, v, 0, kv_len)
        assert np.array_equal(kp, np.asarray(Kp[:, :, :kv_len], np.float32))
        assert np.array_equal(vp, np.asarray(Vp[:, :, :kv_len], np.float32))


@pytest.mark.parametrize("sname,kind,T", [
    ("small_bf16", "ties", 1.0), ("small_bf16", "ties", 0.0), ("ragged_bf16", "ties", 0.7),
    ("small_bf16", "nonfinite", 1.0), ("small_bf16", "nonfinite", 0.0),
    ("ragged_bf16", "nonfinite", 1.3),
])
def test_forward_statistics_special_rows(api, sname, kind, T):
    """The statistics computed with the LM head on logits with ties and
    non-finite values.  ties: every LM-head row zero except rows 100 .. 199,
    which share one vector, so each row of logits is 0 except one value
    repeated 100 times (the largest is tied, its lowest index wins, and the
    1000-odd equal zeros enter the total).  nonfinite: row 7 of the LM head
    +inf, so column 7 of every row is +inf or NaN (the row's total is NaN,
    its argmax ignores NaN)."""
    shape = synth.SHAPES[sname]
    W = dict(weights(shape))
    lm = np.array(W["lm_head"], dtype=np.float32, copy=True)
    if kind == "ties":
        row = lm[100].copy()
        lm[:] = 0.0
        lm[100:200] = row
    else:
        lm[7] = np.inf
    W["lm_head"] = lm
    say(f"forward statistics {sname} {kind} T={T}")
    m = api.Model(shape, api.dict_tensors(W))
    P, parents = 60, synth.branch_parents(3, 4)
    ptoks = synth.prefix_tokens(shape.vocab, P)
    _, Kp, Vp = decoder.prefill(shape, weights(shape), ptoks[:-1], "bf16")
    toks = np.random.default_rng(5).integers(0, shape.vocab, len(parents)).astype(np.int32)
    toks[0] = ptoks[-1]
    st = []
    got, _, _ = gpu_forward(api, m, Kp, Vp, P - 1, toks, parents, T=T, stats_out=st)
    if kind == "ties":
        assert np.all(np.sum(got == got.max(axis=1, keepdims=True), axis=1) >= 100)
    else:
        assert np.all(~np.isfinite(got[:, 7]))
    check_stats(st[0], got, T)


@pytest.mark.parametrize("sname", ["tiny", "small_bf16", "small_gqa_bf16"])
def test_branch_mask_gpu(api, sname):
    """Invariant (a) on the HIP path: each branch's rows in the tree forward
    equal a forward of [root, that branch] alone on the same prefix."""
    shape = synth.SHAPES[sname]
    say(f"branch mask {sname}")
    W = weights(shape)
    B, k = 3, 5
    parents = synth.branch_parents(B, k)
    P = 100
    ptoks = synth.prefix_tokens(shape.vocab, P)
    _, Kp, Vp = decoder.prefill(shape, W, ptoks[:-1], mode(shape))
    g = np.random.default_rng(5)
    toks = g.integers(0, shape.vocab, len(parents)).astype(np.int32)
    toks[0] = ptoks[-1]
    m = model(api, shape)
    lt, _, _ = gpu_forward(api, m, Kp, Vp, P - 1, toks, parents)
    for b in range(B):
        rows = [0] + [1 + b * k + j for j in range(k)]
        lc, _, _ = gpu_forward(api, m, Kp, Vp, P - 1, toks[rows], synth.chain_parents(len(rows)))
        assert row_relerr(lt[rows], lc) < tol(shape) / 4


@pytest.mark.parametrize("sname", ["tiny", "small_bf16"])
def test_gpu_chunked_prefill(api, sname):
    """A prefix built on the GPU by chained verify steps (chain trees of at
    most 64 rows) matches the oracle's prefill."""
    shape = synth.SHAPES[sname]
    say(f"chunked prefill {sname}")
    W = weights(shape)
    P = 150
    ptoks = synth.prefix_tokens(shape.vocab, P)
    _, Kr, Vr = decoder.prefill(shape, W, ptoks, mode(shape))
    m = model(api, shape)
    k, v = m.new_kv(P + 8)
    done = 0
    while done < P:
        n = min(64, P - done)
        logits = torch.empty((n, shape.vocab), dtype=torch.float32, device="cuda")
        stats = api.new_stats(n)
        ws = m.workspace(n, done)
        toks = torch.from_numpy(ptoks[done:done + n].astype(np.int32)).cuda()
        m.sb_verify_forward(k, v, done, toks, synth.chain_parents(n), 1.0, logits, stats, ws)
        done += n
    torch.cuda.synchronize()
    kg, vg = m.read_kv(k, v, 0, P)
    assert row_relerr(kg.reshape(-1, shape.head_dim), Kr.reshape(-1, shape.head_dim)) < tol(shape) * 5
    assert row_relerr(vg.reshape(-1, shape.head_dim), Vr.reshape(-1, shape.head_dim)) < tol(shape) * 5


def test_verify_forward_host_errors(api):
    shape = synth.SHAPES["tiny"]
    m = model(api, shape)
    k, v = m.new_kv(24)
    logits = torch.empty((4, shape.vocab), dtype=torch.float32, device="cuda")
    stats = api.new_stats(4)
    ws = m.workspace(4, 16)
    toks = torch.zeros(4, dtype=torch.int32, device="cuda")
    with pytest.raises(api.SBError) as e:
        m.sb_verify_forward(k, v, 16, toks, [-1, 0, 1, 2], 1.0, logits, stats, ws[:10])
    assert e.value.code == 3           # workspace too small
    with pytest.raises(api.SBError) as e:
        m.sb_verify_forward(k, v, 21, toks, [-1, 0, 1, 2], 1.0, logits, stats, ws)
    assert e.value.code == 3           # kv_len + n_rows > capacity
    with pytest.raises(api.SBError) as e:
        m.sb_verify_forward(k, v, 4, toks, [-1, 0, 3, 1], 1.0, logits, stats, ws)
    assert e.value.code == 2           # parent after child
