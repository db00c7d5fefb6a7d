"""Pin of the oracle rollback (CPU only).

Invariant (c): after a verify step and compaction to the accepted path, the
cache equals a fresh prefill of prefix + root + accepted tokens, and the new
length is P_kv + 1 + n_accepted.  Keeping branch 0 with every draft
accepted leaves the cache untouched.
"""
import numpy as np
import pytest

from oracle import decoder, rollback, sampling
from paper_2506_01979_amd import synth


def _verified_cache(seed_u=1):
    w = synth.WORKLOADS["exact"]
    shape = w.shape
    W = synth.model_weights(shape)
    inp = synth.step_inputs(w, seed_u=seed_u)
    P_kv = w.kv_len
    _, Kp, Vp = decoder.prefill(shape, W, inp["prefix_tokens"][:-1], "f64")
    cap = P_kv + w.n_rows + 4
    K, V = decoder.make_cache(shape, Kp, Vp, P_kv, cap)
    lg, kt, vt = decoder.tree_forward(shape, W, Kp, Vp, P_kv, inp["tokens"], inp["parents"], "f64")
    K, V = decoder.write_tree_kv(K, V, P_kv, kt, vt)
    return w, shape, W, inp, K, V, lg


def _check_fresh_prefill(shape, W, inp, K, V, P_kv, path):
    K2, V2, new_len = rollback.kv_rollback(K, V, P_kv, path)
    assert new_len == P_kv + len(path)
    seq = np.concatenate([inp["prefix_tokens"], [inp["tokens"][i] for i in path[1:]]])
    _, Kf, Vf = decoder.prefill(shape, W, seq, "f64")
    assert np.allclose(K2[:, :, :new_len], Kf, rtol=0, atol=1e-12)
    assert np.allclose(V2[:, :, :new_len], Vf, rtol=0, atol=1e-12)


def test_rollback_equals_fresh_prefill_every_path():
    """Every branch b and every accepted length n = 0..k."""
    w, shape, W, inp, K, V, _ = _verified_cache()
    for b in range(w.branches):
        for n in range(w.depth + 1):
            path = [0] + [1 + b * w.depth + j for j in range(n)]
            _check_fresh_prefill(shape, W, inp, K, V, w.kv_len, path)


@pytest.mark.parametrize("seed_u", [1, 2, 3])
def test_rollback_after_walk(seed_u):
    w, shape, W, inp, K, V, lg = _verified_cache(seed_u)
    r = sampling.accept_resample(inp["tokens"], inp["parents"], lg.astype(np.float32), 1.0,
                                 inp["q"], inp["u"])
    assert len(r.path) == 1 + r.n_accepted
    _check_fresh_prefill(shape, W, inp, K, V, w.kv_len, r.path)


def test_rollback_noop_on_branch_zero():
    shape = synth.SHAPES["exact"]
    g = np.random.default_rng(0)
    K = g.standard_normal((1, 2, 20, 32))
    V = g.standard_normal((1, 2, 20, 32))
    K2, V2, n = rollback.kv_rollback(K, V, 7, [0, 1, 2, 3])
    assert n == 11
    assert np.array_equal(K2, K) and np.array_equal(V2, V)


def test_rollback_reads_before_overwrite():
    """A path whose source slot is a later destination (general trees)."""
    K = np.arange(10, dtype=np.float64).reshape(1, 1, 10, 1)
    V = -K
    # rows: 0 root, 1 child of 0, 2 child of 0, 3 child of 2 -> path [0, 2, 3]
    K2, V2, n = rollback.kv_rollback(K, V, 4, [0, 2, 3])
    assert n == 7
    assert list(K2[0, 0, 4:7, 0]) == [4, 6, 7]
    assert list(V2[0, 0, 4:7, 0]) == [-4, -6, -7]
