"""GPU KV rollback: byte-exact against the oracle compaction on synthetic
cache contents, and invariant (c) end to end -- after verify, accept and
rollback the cache equals a fresh prefill of the accepted sequence.  The
GPU's walk only picks which path is checked; the expected cache of a path
comes from the oracle's prefill of the prefix and that path's draft tokens,
both seeded inputs."""
import numpy as np
import pytest
import torch

from gpu_util import row_relerr, say
from oracle import decoder, rollback, sampling
from paper_2506_01979_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def api():
    from paper_2506_01979_amd import api as A
    assert torch.cuda.is_available()
    return A


def result_tensor(api, path):
    a = np.full(api.STEP_RESULT_INTS, -1, dtype=np.int32)
    a[0] = len(path) - 1
    a[3] = len(path)
    a[8:8 + len(path)] = path
    return torch.from_numpy(a).cuda()


@pytest.mark.parametrize("sname", ["tiny", "small_bf16", "small_gqa_bf16"])
@pytest.mark.parametrize("path", [[0, 1, 2, 3], [0, 9, 10, 11], [0, 2, 3], [0], [0, 17, 18],
                                  list(range(64)), [0, 128, 200, 255]])
def test_rollback_bytes(api, sname, path):
    shape = synth.SHAPES[sname]
    say(f"rollback bytes {sname} path={path}")
    m = api.Model(shape.with_layers(2), api.synth_tensors(shape.with_layers(2)))
    # rows up to 255 of a 256-row tree behind the prefix
    kv_len, cap = 37, max(80, (37 + max(path) + 1 + 7) // 8 * 8)
    g = np.random.default_rng(len(path))
    L = 2
    K = g.standard_normal((L, shape.n_kv_heads, cap, shape.head_dim)).astype(np.float32)
    V = g.standard_normal((L, shape.n_kv_heads, cap, shape.head_dim)).astype(np.float32)
    if shape.dtype == "bf16":
        K = decoder.round_bf16(K)
        V = decoder.round_bf16(V)
    k, v = m.new_kv(cap)
    m.load_kv(k, v, K, V, cap)
    new_len = torch.zeros(1, dtype=torch.int32, device="cuda")
    m.sb_kv_rollback(k, v, kv_len, result_tensor(api, path), new_len)
    torch.cuda.synchronize()
    K2, V2, n2 = rollback.kv_rollback(K, V, kv_len, path)
    assert int(new_len.item()) == n2
    kg, vg = m.read_kv(k, v, 0, cap)
    assert np.array_equal(kg, K2)
    assert np.array_equal(vg, V2)


@pytest.mark.parametrize("sname,seed_u", [("tiny", 1), ("tiny", 4), ("small_bf16", 2),
                                          ("small_bf16", 3)])
def test_rollback_equals_fresh_prefill(api, sname, seed_u):
    shape = synth.SHAPES[sname]
    say(f"rollback end-to-end {sname} seed_u={seed_u}")
    W = synth.model_weights(shape)
    md = "bf16" if shape.dtype == "bf16" else "f64"
    tol = 2e-2 if shape.dtype == "bf16" else 1e-4
    B, kk, P = 3, 4, 60
    parents = synth.branch_parents(B, kk)
    n = len(parents)
    ptoks = synth.prefix_tokens(shape.vocab, P)
    kv_len = P - 1
    _, Kp, Vp = decoder.prefill(shape, W, ptoks[:-1], md)
    m = api.Model(shape, api.dict_tensors(W))
    cap = kv_len + n + 4
    k, v = m.new_kv(cap)
    m.load_kv(k, v, Kp, Vp, kv_len)
    g = np.random.default_rng(seed_u)
    toks = g.integers(0, shape.vocab, n).astype(np.int32)
    toks[0] = ptoks[-1]
    logits = torch.empty((n, shape.vocab), dtype=torch.float32, device="cuda")
    stats = api.new_stats(n)
    ws = m.workspace(n, kv_len)
    tt = torch.from_numpy(toks).cuda()
    m.sb_verify_forward(k, v, kv_len, tt, parents, 1.0, logits, stats, ws)
    # q aligned with the target rows of the parents makes long paths likely
    lg = logits.cpu().numpy()
    q = np.zeros((n, shape.vocab), dtype=np.float32)
    for i in range(1, n):
        p = sampling.target_probs(lg[parents[i]], 1.0)
        q[i] = (0.9 * p + 0.1 / shape.vocab).astype(np.float32)
    u = synth.uniforms(n, seed_u)
    res = api.new_result()
    sws = torch.empty(api.sb_sample_workspace_bytes(shape.vocab), dtype=torch.uint8, device="cuda")
    api.sb_accept_resample(tt, parents, logits, stats, 1.0, torch.from_numpy(q).cuda(),
                           torch.from_numpy(u).cuda(), res, sws)
    new_len = torch.zeros(1, dtype=torch.int32, device="cuda")
    m.sb_kv_rollback(k, v, kv_len, res, new_len)
    torch.cuda.synchronize()
    r = api.decode_result(res)
    nl = int(new_len.item())
    assert nl == kv_len + 1 + r["n_accepted"]
    path = r["path"]
    assert path in expected_paths(B, kk)
    # expected cache of every possible accepted path, from the oracle alone
    acc = [int(toks[i]) for i in path[1:]]
    seq = np.concatenate([ptoks, np.asarray(acc, np.int32)])
    _, Kf, Vf = decoder.prefill(shape, W, seq, md)
    kg, vg = m.read_kv(k, v, 0, nl)
    assert row_relerr(kg.reshape(-1, shape.head_dim), Kf.reshape(-1, shape.head_dim)) < 5 * tol
    assert row_relerr(vg.reshape(-1, shape.head_dim), Vf.reshape(-1, shape.head_dim)) < 5 * tol
    # the same rows from a fresh GPU forward of root + accepted tokens
    k2, v2 = m.new_kv(cap)
    k2[:, :, :kv_len] = k[:, :, :kv_len]
    v2[:, :, :, :kv_len] = v[:, :, :, :kv_len]
    nn = 1 + len(acc)
    l2 = torch.empty((nn, shape.vocab), dtype=torch.float32, device="cuda")
    m.sb_verify_forward(k2, v2, kv_len, torch.from_numpy(seq[kv_len:].astype(np.int32)).cuda(),
                        synth.chain_parents(nn), 1.0, l2, api.new_stats(nn), m.workspace(nn, kv_len))
    torch.cuda.synchronize()
    k2g, _ = m.read_kv(k2, v2, 0, nl)
    assert row_relerr(k2g.reshape(-1, shape.head_dim), kg.reshape(-1, shape.head_dim)) < tol


def expected_paths(B, k):
    """Every path the walk may keep in a B x k branch tree."""
    out = [[0]]
    for b in range(B):
        for n in range(1, k + 1):
            out.append([0] + [1 + b * k + j for j in range(n)])
    return out
