"""GPU parity of the persistent forward (one cooperative launch for every
layer, SB_FWD_PERSISTENT) against the oracle, and against the chain of
kernels (SB_FWD_KERNELS) on the same inputs.

Cases cover 1..4 token tiles (5, 17, 33, 64 rows), multi-head and grouped
queries at head width 128, a branch tree, a chain and the chain-plus-fork
shape, an empty-looking prefix (one slot) and prefixes whose key ranges give
several attention items per workgroup (13B width, prefix 8192).  Logits are
held to the bf16 bound 2e-2 per row against the oracle's bf16 emulation,
the tree K/V to 5 times that, the prefix slots must be untouched and two
runs must agree bit for bit (the forward is deterministic)."""
import numpy as np
import pytest
import torch

from gpu_util import row_relerr, say
from oracle import decoder, sampling
from paper_2506_01979_amd import synth

pytestmark = pytest.mark.gpu

TOL = 2e-2


@pytest.fixture(scope="module")
def api():
    from paper_2506_01979_amd import api as A
    assert torch.cuda.is_available()
    return A


_W, _M = {}, {}


def model(api, shape):
    if shape.name not in _M:
        _W[shape.name] = synth.model_weights(shape)
        _M[shape.name] = api.Model(shape, api.dict_tensors(_W[shape.name]))
    return _M[shape.name], _W[shape.name]


def tree_of(spec):
    if spec[0] == "branch":
        return synth.branch_parents(spec[1], spec[2])
    if spec[0] == "fork":
        return synth.fork_parents(spec[1], spec[2], spec[3])
    return synth.chain_parents(spec[1])


def run(api, m, mode, Kp, Vp, kv_len, toks, parents):
    n = len(parents)
    m.sb_model_set_forward(mode)
    k, v = m.new_kv(kv_len + n + 8)
    if kv_len:
        m.load_kv(k, v, Kp, Vp, kv_len)
    logits = torch.full((n, m.shape.vocab), float("nan"), dtype=torch.float32, device="cuda")
    stats = api.new_stats(n)
    m.sb_verify_forward(k, v, kv_len, torch.from_numpy(toks).cuda(), parents, 1.0, logits, stats,
                        m.workspace(n, kv_len))
    torch.cuda.synchronize()
    m.sb_model_set_forward(api.SB_FWD_AUTO)
    return logits.cpu().numpy(), api.decode_stats(stats), k, v


CASES = [
    ("small_h128_bf16", 200, ("branch", 4, 8)),   # 33 rows, 3 token tiles
    ("small_h128_bf16", 64, ("branch", 1, 4)),    # 5 rows, 1 tile
    ("small_h128_bf16", 300, ("branch", 4, 4)),   # 17 rows, 2 tiles
    ("small_h128_bf16", 90, ("chain", 64)),       # 64 rows, 4 tiles
    ("small_h128_bf16", 2, ("fork", 4, 4, 7)),    # one prefix slot; chain + fork
    ("small_gqa128_bf16", 300, ("branch", 4, 8)), # grouped queries, 8 per KV head
    ("small_gqa128_bf16", 33, ("branch", 2, 3)),
]


@pytest.mark.parametrize("sname,P,spec", CASES, ids=[f"{c[0]}-P{c[1]}-{c[2]}" for c in CASES])
def test_persistent_forward_parity(api, sname, P, spec):
    shape = synth.SHAPES[sname]
    m, W = model(api, shape)
    parents = tree_of(spec)
    n = len(parents)
    kv_len = P - 1
    ptoks = synth.prefix_tokens(shape.vocab, P)
    _, Kp, Vp = decoder.prefill(shape, W, ptoks[:-1], "bf16")
    g = np.random.default_rng(P + n)
    toks = g.integers(0, shape.vocab, n).astype(np.int32)
    toks[0] = ptoks[-1]
    ref, kt, vt = decoder.tree_forward(shape, W, Kp, Vp, kv_len, toks, parents, "bf16")
    say(f"persistent forward {sname} P={P} tree={spec} ({n} rows)")
    lp, sp, k, v = run(api, m, api.SB_FWD_PERSISTENT, Kp, Vp, kv_len, toks, parents)
    err = row_relerr(lp, ref)
    say(f"  logits row-relative error {err:.3e}")
    assert np.all(np.isfinite(lp)) and err < TOL
    kg, vg = m.read_kv(k, v, kv_len, n)
    assert row_relerr(kg.reshape(-1, shape.head_dim), kt.reshape(-1, shape.head_dim)) < 5 * TOL
    assert row_relerr(vg.reshape(-1, shape.head_dim), vt.reshape(-1, shape.head_dim)) < 5 * TOL
    kp, vp = m.read_kv(k, v, 0, kv_len)
    assert np.array_equal(kp, np.asarray(Kp[:, :, :kv_len], np.float32))
    assert np.array_equal(vp, np.asarray(Vp[:, :, :kv_len], np.float32))
    for i in range(n):
        rs = sampling.row_stats(lp[i], 1.0)
        assert sp[i]["argmax"] == rs.argmax and sp[i]["zmax"] == np.float32(rs.zmax)
        assert abs(sp[i]["total"] - rs.total) <= 1e-6 * rs.total
    # deterministic, and the kernel chain agrees with the oracle as well
    lp2, _, _, _ = run(api, m, api.SB_FWD_PERSISTENT, Kp, Vp, kv_len, toks, parents)
    assert np.array_equal(lp.view(np.uint32), lp2.view(np.uint32))
    lk, _, _, _ = run(api, m, api.SB_FWD_KERNELS, Kp, Vp, kv_len, toks, parents)
    say(f"  kernel chain error {row_relerr(lk, ref):.3e}, persistent vs chain {row_relerr(lp, lk):.3e}")
    assert row_relerr(lk, ref) < TOL


def test_persistent_rejects_what_it_does_not_fit(api):
    """Head width 64 and more than 64 rows are outside the persistent
    kernel: SB_FWD_PERSISTENT returns SB_ERR_UNSUPPORTED; AUTO runs the
    chain."""
    shape = synth.SHAPES["small_bf16"]
    m, W = model(api, shape)
    parents = synth.branch_parents(2, 4)
    toks = np.arange(len(parents), dtype=np.int32)
    with pytest.raises(api.SBError):
        run(api, m, api.SB_FWD_PERSISTENT, None, None, 0, toks, parents)
    shape = synth.SHAPES["small_h128_bf16"]
    m, W = model(api, shape)
    parents = synth.branch_parents(8, 16)  # 129 rows
    toks = np.arange(len(parents), dtype=np.int32) % shape.vocab
    with pytest.raises(api.SBError):
        run(api, m, api.SB_FWD_PERSISTENT, None, None, 0, toks, parents)
    lg, _, _, _ = run(api, m, api.SB_FWD_AUTO, None, None, 0, toks, parents)
    assert np.all(np.isfinite(lg))


@pytest.mark.timeout(600)
def test_persistent_13b_slice_long_prefix(api):
    """13B width (40 KV heads), prefix 8192: 17 key ranges per head, 680
    attention items over the workgroups (several per workgroup)."""
    shape = synth.SHAPES["llama13b"].with_layers(2)
    say("persistent 13B slice, prefix 8192, tree 4x8")
    W = synth.model_weights(shape)
    m = api.Model(shape, api.dict_tensors(W))
    P, parents = 8192, synth.branch_parents(4, 8)
    n, kv_len = len(parents), 8191
    Kp = np.stack([synth.synthetic_kv(shape, l, kv_len, kv_len, 0) for l in range(2)])
    Vp = np.stack([synth.synthetic_kv(shape, l, kv_len, kv_len, 1) for l in range(2)])
    toks = np.random.default_rng(3).integers(0, shape.vocab, n).astype(np.int32)
    ref, _, _ = decoder.tree_forward(shape, W, Kp, Vp, kv_len, toks, parents, "bf16")
    lp, _, _, _ = run(api, m, api.SB_FWD_PERSISTENT, Kp, Vp, kv_len, toks, parents)
    err = row_relerr(lp, ref)
    say(f"  logits row-relative error {err:.3e}")
    assert err < TOL
