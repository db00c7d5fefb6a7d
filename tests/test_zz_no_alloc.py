"""The verify forward without a workspace argument (sb_verify_forward_noalloc,
for callers that cannot allocate): its scratch array must give exactly what
the workspace entry point gives, on calls in a row each smaller than the
one before (the array keeps the previous call's contents)."""
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


def _inputs(shape, P, B, k, seed):
    g = np.random.default_rng(seed)
    parents = synth.branch_parents(B, k)
    toks = g.integers(0, shape.vocab, len(parents)).astype(np.int32)
    return parents, toks


def _fill_prefix(m, k, v, kv_len, seed):
    g = torch.Generator(device="cpu").manual_seed(seed)
    kk = torch.randn(k[:, :, :kv_len].shape, generator=g).to(torch.bfloat16)
    vv = torch.randn(v[:, :, :, :kv_len].shape, generator=g).to(torch.bfloat16)
    k[:, :, :kv_len] = kk.cuda()
    v[:, :, :, :kv_len] = vv.cuda()


@pytest.mark.parametrize("sname", ["small_bf16", "small_gqa_bf16"])
def test_noalloc_equals_workspace_entry(api, sname):
    shape = synth.SHAPES[sname]
    W = synth.model_weights(shape)
    m = api.Model(shape, api.dict_tensors(W))
    # a wide tree (129 rows: the wide GEMMs and LM head), then smaller ones
    for call, (P, B, k) in enumerate(((300, 8, 16), (300, 4, 8), (40, 2, 3))):
        kv_len = P - 1
        parents, toks = _inputs(shape, P, B, k, 10 + call)
        n = len(parents)
        say(f"no-alloc forward {sname} call {call}: prefix {P}, tree {B}x{k} ({n} rows)")
        out = []
        for entry in ("workspace", "noalloc"):
            kc, vc = m.new_kv(kv_len + n + 8)
            _fill_prefix(m, kc, vc, kv_len, 100 + call)
            logits = torch.full((n, shape.vocab), float("nan"), dtype=torch.float32, device="cuda")
            stats = api.new_stats(n)
            d_tok = torch.from_numpy(toks).cuda()
            if entry == "workspace":
                m.sb_verify_forward(kc, vc, kv_len, d_tok, parents, 1.0, logits, stats,
                                    m.workspace(n, kv_len))
            else:
                m.sb_verify_forward_noalloc(kc, vc, kv_len, d_tok, parents, 1.0, logits, stats)
            torch.cuda.synchronize()
            out.append((logits.cpu().numpy(), stats.cpu().numpy(), kc.cpu(), vc.cpu()))
        (l0, s0, k0, v0), (l1, s1, k1, v1) = out
        assert np.all(np.isfinite(l0))
        assert np.array_equal(l0.view(np.uint32), l1.view(np.uint32))
        assert np.array_equal(s0, s1)
        assert torch.equal(k0.view(torch.int16), k1.view(torch.int16))
        assert torch.equal(v0.view(torch.int16), v1.view(torch.int16))
