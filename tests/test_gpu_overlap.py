"""Algorithm 2's drafting/verification overlap on one GPU.

The target's verify step (forward, accept/resample walk, rollback) runs on
one stream while the draft builds the next round's branches
(sb_draft_round) on another, then Algorithm 1 (sb_select_branch) tests the
branches' first tokens at a row of the verified tree.  Overlap changes only
the schedule: every output -- logits, statistics, the walk's result, the
rolled-back cache length, the draft's tokens and q rows, the selection --
must equal the serial run's bit for bit, on every repetition.  Each piece's
parity against the oracle is covered by its own tests.
"""
import numpy as np
import pytest
import torch

from gpu_util import say
from paper_2506_01979_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def api():
    from paper_2506_01979_amd import api as A
    assert torch.cuda.is_available()
    return A


def test_overlapped_round_equals_serial(api):
    dev = "cuda"
    tshape = synth.SHAPES["small_bf16"]
    dshape = synth.SHAPES["small_bf16"]
    tm = api.Model(tshape, api.synth_tensors(tshape, seed=0))
    dm = api.Model(dshape, api.synth_tensors(dshape, seed=1))
    P, B, kd = 300, 4, 8
    parents = synth.branch_parents(B, kd)
    n = len(parents)
    V = tshape.vocab

    def prefix(m, shp):
        k, v = m.new_kv(P + n + 16)
        K = np.stack([synth.synthetic_kv(shp, li, P, P, 0, as_bits=True)
                      for li in range(shp.n_layers)])
        Vv = np.stack([synth.synthetic_kv(shp, li, P, P, 1, as_bits=True)
                       for li in range(shp.n_layers)])
        m.load_kv(k, v, K, Vv, P)
        return k, v
    tk, tv = prefix(tm, tshape)
    dk, dv = prefix(dm, dshape)
    q = synth.draft_q(n, V, 0.7, seed=3)
    toks = torch.from_numpy(synth.draw_tokens(q, seed=3)).to(dev)
    toks[0] = 5
    qd = torch.from_numpy(q).to(dev)
    ud = torch.from_numpy(synth.uniforms(n, 4)).to(dev)
    logits = torch.empty((n, V), dtype=torch.float32, device=dev)
    stats = api.new_stats(n)
    ws = tm.workspace(n, P)
    sws = torch.empty(api.sb_sample_workspace_bytes(V), dtype=torch.uint8, device=dev)
    res = api.new_result()
    new_len = torch.zeros(1, dtype=torch.int32, device=dev)
    K_MAX, DEPTH = 4, 8
    R = 1 + K_MAX * DEPTH
    du = torch.from_numpy(synth.uniforms(R, 5)).to(dev)
    dtok = torch.full((R,), 9, dtype=torch.int32, device=dev)
    dq = torch.zeros((R, V), dtype=torch.float32, device=dev)
    dws = dm.draft_round_workspace(K_MAX, DEPTH, P)
    su = torch.from_numpy(synth.uniforms(K_MAX + 1, 6)).to(dev)
    sel = torch.empty(3, dtype=torch.int32, device=dev)
    cur = torch.cuda.current_stream()

    def verify(st):
        tm.sb_verify_forward(tk, tv, P, toks, parents, 1.0, logits, stats, ws, st)
        api.sb_accept_resample(toks, parents, logits, stats, 1.0, qd, ud, res, sws, st)
        tm.sb_kv_rollback(tk, tv, P, res, new_len, st)

    def outputs(nb):
        return (logits.cpu().numpy().copy(), stats.cpu().numpy().copy(), api.decode_result(res),
                int(new_len.item()), nb, dtok.cpu().numpy().copy(), dq.cpu().numpy().copy(),
                sel.cpu().tolist())

    say("overlap: serial round")
    verify(cur)
    nb, _, _ = dm.sb_draft_round(dk, dv, P, K_MAX, "wor", DEPTH, 1.0, du, dtok, dq, dws, cur)
    api.sb_select_branch(logits[n - 1], stats[n - 1], 1.0, dtok[1:1 + nb], dq[1:1 + nb], su, sel,
                         sws, cur)
    torch.cuda.synchronize()
    want = outputs(nb)
    sv, sd = torch.cuda.Stream(), torch.cuda.Stream()
    for rep in range(3):
        say(f"overlap: two-stream round {rep}")
        logits.zero_()
        dq.zero_()
        torch.cuda.synchronize()
        sv.wait_stream(cur)
        sd.wait_stream(cur)
        verify(sv)
        nb2, _, _ = dm.sb_draft_round(dk, dv, P, K_MAX, "wor", DEPTH, 1.0, du, dtok, dq, dws, sd)
        cur.wait_stream(sv)
        cur.wait_stream(sd)
        api.sb_select_branch(logits[n - 1], stats[n - 1], 1.0, dtok[1:1 + nb2], dq[1:1 + nb2], su,
                             sel, sws, cur)
        torch.cuda.synchronize()
        got = outputs(nb2)
        assert np.array_equal(got[0], want[0]) and np.array_equal(got[1], want[1])
        assert got[2:5] == want[2:5]
        assert np.array_equal(got[5], want[5]) and np.array_equal(got[6], want[6])
        assert got[7] == want[7]
