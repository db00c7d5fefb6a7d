"""CPU checks of the C ABI: the library loads, exports every entry point
that include/sb.h declares, and rejects bad arguments on the host before
anything reaches a device."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sb.h")


def declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(sb_[a-z_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def api():
    from paper_2506_01979_amd import api as A
    return A


def test_exports_every_declared_symbol(api):
    names = declared()
    assert len(names) >= 13
    for n in names:
        assert hasattr(api.lib, n), n
    assert set(api.EXPORTS) == set(names)


def test_version_and_strings(api):
    assert api.lib.sb_version() == 1
    for code in range(7):
        assert api.lib.sb_status_string(code)


def cfg(api, **kw):
    from paper_2506_01979_amd import synth
    c = api.make_config(synth.SHAPES["llama7b"])
    for k, v in kw.items():
        setattr(c, k, v)
    return c


def test_packed_bytes(api):
    c = cfg(api)
    # 7B shape: QKV 12288 x 4096, O 4096 x 4096, gate/up 2 x 11008 x 4096,
    # down 4096 x 11008, LM head 32000 x 4096 -- bf16, no padding needed
    assert api.sb_packed_bytes(c, api.SB_W_QKV) == 12288 * 4096 * 2
    assert api.sb_packed_bytes(c, api.SB_W_O) == 4096 * 4096 * 2
    assert api.sb_packed_bytes(c, api.SB_W_GATE_UP) == 2 * 11008 * 4096 * 2
    assert api.sb_packed_bytes(c, api.SB_W_DOWN) == 4096 * 11008 * 2
    assert api.sb_packed_bytes(c, api.SB_W_LM_HEAD) == 32000 * 4096 * 2
    assert api.sb_packed_bytes(c, 9) == 0
    bad = cfg(api, n_kv_heads=5)
    assert api.sb_packed_bytes(bad, api.SB_W_QKV) == 0
    # ragged ffn (688) is padded to whole 256-column chunks, vocab (1000)
    # to whole 16-row tiles; gate/up rows cover the padded ffn columns
    from paper_2506_01979_amd import synth
    s = api.make_config(synth.SHAPES["small_bf16"])
    assert api.sb_packed_bytes(s, api.SB_W_DOWN) == 256 * 768 * 2
    assert api.sb_packed_bytes(s, api.SB_W_GATE_UP) == 2 * 768 * 256 * 2
    assert api.sb_packed_bytes(s, api.SB_W_LM_HEAD) == 1008 * 256 * 2


def test_host_validation_without_device(api):
    lib = api.lib
    c = cfg(api)
    h = C.c_void_p()
    assert lib.sb_model_create(C.byref(c), None, C.byref(h)) == 1
    assert lib.sb_model_create(None, None, C.byref(h)) == 1
    bad = cfg(api, head_dim=96)
    w = api.ModelWeights(1, 1, 1, (api.LayerWeights * 32)())
    assert lib.sb_model_create(C.byref(bad), C.byref(w), C.byref(h)) == 6
    assert lib.sb_workspace_bytes(None, 4, 10) == 0
    kv = api.KVCache(1, 1, 100)
    par = (C.c_int32 * 3)(-1, 0, 1)
    assert lib.sb_verify_forward(None, C.byref(kv), 10, 1, par, 3, 1.0, 1, 1, 1, 10, None) == 1
    assert lib.sb_softmax_stats(0, 1, 1, 1.0, 1, None) == 1
    assert lib.sb_softmax_stats(10, 1, 1, -1.0, 1, None) == 1
    bad_par = (C.c_int32 * 3)(-1, 0, 2)
    assert lib.sb_accept_resample(10, 3, 1, bad_par, 1, 1, 1.0, 1, 1, 1, 1, 1 << 20, None) == 2
    root_par = (C.c_int32 * 2)(0, 0)
    assert lib.sb_accept_resample(10, 2, 1, root_par, 1, 1, 1.0, 1, 1, 1, 1, 1 << 20, None) == 2
    assert lib.sb_accept_resample(10, 3, 1, par, 1, 1, 1.0, 1, 1, 1, 1, 8, None) == 3
    assert lib.sb_select_branch(10, 1, 1, 1.0, 0, 1, 1, 1, 1, 1, 1 << 20, None) == 1
    assert lib.sb_kv_rollback(None, C.byref(kv), 3, 1, 1, None) == 1
    assert lib.sb_sample_workspace_bytes(1000) == 16000


def test_hrad_host_validation_without_device(api):
    """H-RAD's tap and predictor reject bad arguments before any launch; a
    model record needs no device (sb_model_create keeps the pointers)."""
    lib = api.lib
    w = api.ModelWeights(1, 1, 1, (api.LayerWeights * 2)(*[api.LayerWeights(1, 1, 1, 1, 1, 1)] * 2))
    h16, h32 = C.c_void_p(), C.c_void_p()
    assert lib.sb_model_create(C.byref(cfg(api, n_layers=2, dtype=api.SB_BF16)), C.byref(w), C.byref(h16)) == 0
    assert lib.sb_model_create(C.byref(cfg(api, n_layers=2, dtype=api.SB_F32)), C.byref(w), C.byref(h32)) == 0
    try:
        assert lib.sb_model_set_tap(None, 1, 1, 4) == 1
        assert lib.sb_model_set_tap(h32, 1, 1, 4) == 4          # float32 models: no tap
        assert lib.sb_model_set_tap(h16, 1, 0, 4) == 1          # k outside 1..n_layers
        assert lib.sb_model_set_tap(h16, 1, 3, 4) == 1
        assert lib.sb_model_set_tap(h16, 1, 2, 257) == 1        # rows outside 1..SB_MAX_ROWS
        assert lib.sb_model_set_tap(h16, 1, 2, 4) == 0
        assert lib.sb_model_set_tap(h16, None, 0, 0) == 0       # cleared
        assert lib.sb_hrad_workspace_bytes() == 1024
        hw = api.HradWeights(1, 1, 1, 1, 1, 1)
        args = lambda m, k=2, rows=4, ws=1024, hwp=C.byref(hw): (m, 1, k, rows, 1, hwp, 1, 1, 1, ws, None)
        assert lib.sb_hrad_predict(*args(None)) == 1
        assert lib.sb_hrad_predict(*args(h32)) == 4
        assert lib.sb_hrad_predict(*args(h16, k=3)) == 1
        assert lib.sb_hrad_predict(*args(h16, ws=512)) == 3
        assert lib.sb_hrad_predict(*args(h16, hwp=C.byref(api.HradWeights(1, 1, 1, None, 1, 1)))) == 1
    finally:
        lib.sb_model_destroy(h16)
        lib.sb_model_destroy(h32)


def test_branch_candidates_host_validation_without_device(api):
    """Branch-point candidates reject bad arguments before any launch (the
    pointers are never dereferenced on these paths)."""
    lib = api.lib
    assert lib.sb_branch_workspace_bytes() >= 8 * api.SB_BRANCH_MAX_K

    def call(q=1, vocab=1000, x_b=1, k_max=6, mode=2, u=1, count=1, toks=1, rows=1, ws=1,
             ws_bytes=None):
        wb = lib.sb_branch_workspace_bytes() if ws_bytes is None else ws_bytes
        return lib.sb_branch_candidates(q, vocab, x_b, k_max, mode, u, count, toks, rows, ws, wb,
                                        None)
    assert call(q=None) == 1
    assert call(rows=None) == 1
    assert call(ws=None) == 1
    assert call(mode=3) == 1
    assert call(mode=-1) == 1
    assert call(u=None) == 1                      # draws need uniforms ...
    assert call(mode=1, u=None) == 1
    assert call(x_b=None) == 1
    assert call(k_max=0) == 1
    assert call(k_max=api.SB_BRANCH_MAX_K + 1) == 1
    assert call(vocab=0) == 1
    assert call(vocab=api.SB_BRANCH_MAX_VOCAB + 1) == 1
    assert call(ws_bytes=8) == 3


def test_draft_host_validation_without_device(api):
    """The draft sampler and the draft round reject bad arguments before any
    launch; the round's workspace size is host arithmetic."""
    lib = api.lib
    I = lambda *a: (C.c_int32 * len(a))(*a)

    def samp(n=2, src=(0, 1), dst=(0, 1), nl=2, no=2, T=1.0, logits=1, u=1, ws=1, wb=None):
        wb = lib.sb_draft_sample_workspace_bytes(100, n) if wb is None else wb
        return lib.sb_draft_sample(100, n, logits, 1, nl, I(*src), T, u, 1, 1, no, I(*dst), ws, wb,
                                   None)
    assert lib.sb_draft_sample_workspace_bytes(100, 2) == 2 * 8
    assert lib.sb_draft_sample_workspace_bytes(4097, 3) == 3 * 3 * 8     # blocks of 2048
    assert lib.sb_draft_sample_workspace_bytes(100, 0) == 0
    assert samp(ws=None) == 1
    assert samp(wb=15) == 3
    assert samp(logits=None) == 1
    assert samp(u=None) == 1
    assert samp(n=0) == 1
    assert samp(n=api.SB_DRAFT_MAX_ROWS + 1, src=(0,) * 65, dst=tuple(range(65)), no=65) == 1
    assert samp(src=(0, 2)) == 1                       # source row past the logits
    assert samp(dst=(0, 2)) == 1                       # destination past the outputs
    assert samp(dst=(1, 1)) == 1                       # two rows into one destination
    assert samp(T=-1.0) == 1
    assert samp(T=float("nan")) == 1
    w = api.ModelWeights(1, 1, 1, (api.LayerWeights * 2)(*[api.LayerWeights(1, 1, 1, 1, 1, 1)] * 2))
    h = C.c_void_p()
    assert lib.sb_model_create(C.byref(cfg(api, n_layers=2, dtype=api.SB_BF16)), C.byref(w), C.byref(h)) == 0
    try:
        assert lib.sb_draft_round_workspace_bytes(None, 6, 4, 1, 100) == 0
        assert lib.sb_draft_round_workspace_bytes(h, 0, 4, 1, 100) == 0
        assert lib.sb_draft_round_workspace_bytes(h, 17, 4, 1, 100) == 0
        assert lib.sb_draft_round_workspace_bytes(h, 6, 4, 0, 100) == 0
        assert lib.sb_draft_round_workspace_bytes(h, 16, 16, 1, 100) == 0   # 257 rows
        assert lib.sb_draft_round_workspace_bytes(h, 16, 15, 17, 100) == 0  # 257 rows
        wb = lib.sb_draft_round_workspace_bytes(h, 6, 4, 1, 100)
        assert wb > 0
        kv = api.KVCache(1, 1, 128)
        par = (C.c_int32 * 32)()
        nb, nc = C.c_int32(0), C.c_int32(0)

        def rnd(m=h, mode=2, k_max=6, depth=4, trunk=1, conf=0.5, cap=128, ws=wb, T=1.0, u=1):
            kv.capacity = cap
            return lib.sb_draft_round(m, C.byref(kv), 100, k_max, mode, depth, trunk, conf, T, u, 1,
                                      1, par, C.byref(nb), C.byref(nc), 1, ws, None)
        assert rnd(m=None) == 1
        assert rnd(u=None) == 1
        assert rnd(mode=5) == 1
        assert rnd(k_max=0) == 1
        assert rnd(depth=0) == 1
        assert rnd(trunk=0) == 1
        assert rnd(conf=float("nan")) == 1
        assert rnd(T=-0.5) == 1
        assert rnd(ws=wb - 1) == 3
        assert rnd(cap=120) == 3                        # 100 + 25 slots needed
    finally:
        lib.sb_model_destroy(h)


def test_noalloc_rejects_a_step_larger_than_its_scratch_without_device(api):
    """sb_verify_forward_noalloc checks the step's workspace against its
    scratch array before any device call: a 70B-shaped step of 256 rows at
    a 60000-slot prefix needs more than 128 MiB."""
    lib = api.lib
    w = api.ModelWeights(1, 1, 1, (api.LayerWeights * 2)(*[api.LayerWeights(1, 1, 1, 1, 1, 1)] * 2))
    from paper_2506_01979_amd import synth
    c = api.make_config(synth.SHAPES["llama70b"].with_layers(2))
    h = C.c_void_p()
    assert lib.sb_model_create(C.byref(c), C.byref(w), C.byref(h)) == 0
    try:
        assert lib.sb_workspace_bytes(h, 256, 60000) > api.SB_NOALLOC_SCRATCH_BYTES
        kv = api.KVCache(1, 1, 65536)
        par = (C.c_int32 * 256)(*([-1] + list(range(255))))
        assert lib.sb_verify_forward_noalloc(h, C.byref(kv), 60000, 1, par, 256, 1.0, 1, 1,
                                             None) == 3
        assert lib.sb_verify_forward_noalloc(None, C.byref(kv), 60000, 1, par, 256, 1.0, 1, 1,
                                             None) == 1
    finally:
        lib.sb_model_destroy(h)


def _fake_model(api, shape_name, n_layers=None):
    """A model handle over placeholder weight pointers (host arithmetic only:
    nothing here launches)."""
    from paper_2506_01979_amd import synth
    sh = synth.SHAPES[shape_name]
    L = n_layers or sh.n_layers
    w = api.ModelWeights(1, 1, 1, (api.LayerWeights * L)(*[api.LayerWeights(1, 1, 1, 1, 1, 1)] * L))
    c = api.make_config(sh.with_layers(L) if n_layers else sh)
    h = C.c_void_p()
    assert api.lib.sb_model_create(C.byref(c), C.byref(w), C.byref(h)) == 0
    return h, w


@pytest.mark.parametrize("shape,rows,prefixes", [
    ("llama7b", 129, (512, 2048, 4096, 8192)),
    ("llama13b", 129, (512, 2048, 4096, 8192)),
    ("llama13b", 65, (8192,)),
    ("llama70b", 33, (512, 4096, 8192)),
])
def test_noalloc_scratch_covers_the_stated_steps(api, shape, rows, prefixes):
    """The allocation-free entry point's 128 MiB array holds the forward's
    workspace of the steps its documentation names."""
    h, _w = _fake_model(api, shape)
    try:
        for P in prefixes:
            assert 0 < api.lib.sb_workspace_bytes(h, rows, P - 1) <= api.SB_NOALLOC_SCRATCH_BYTES
    finally:
        api.lib.sb_model_destroy(h)


def test_round_host_validation_without_device(api):
    """sb_round_finish and sb_spec_round reject bad arguments before any
    launch; the round's workspace size is host arithmetic."""
    lib = api.lib
    # sb_round_finish: null buffers, negative counts, too many rows, no
    # selection with candidates
    assert lib.sb_round_finish(2, 3, 4, None, 1, 1, 1, None) == 1
    assert lib.sb_round_finish(2, 3, 4, 1, None, 1, 1, None) == 1
    assert lib.sb_round_finish(-1, 3, 4, 1, 1, 1, 1, None) == 1
    assert lib.sb_round_finish(2, 3, 0, 1, 1, 1, 1, None) == 1
    assert lib.sb_round_finish(10, 16, 16, 1, 1, 1, 1, None) == 1     # 1 + 10 + 256 rows
    t, _wt = _fake_model(api, "small_bf16")
    d, _wd = _fake_model(api, "small_bf16")
    try:
        p = api.RoundParams(4, 2, 3, 4, 0.1, 1.0, 0)
        wb = lib.sb_spec_round_workspace_bytes(t, d, C.byref(p), 100, 100)
        assert wb > 0
        assert lib.sb_spec_round_workspace_bytes(t, None, C.byref(p), 100, 100) == 0
        bad = api.RoundParams(0, 2, 3, 4, 0.1, 1.0, 0)
        assert lib.sb_spec_round_workspace_bytes(t, d, C.byref(bad), 100, 100) == 0
        tkv, dkv = api.KVCache(1, 1, 128), api.KVCache(1, 1, 128)
        par = (C.c_int32 * 64)()
        nc, nb = C.c_int32(0), C.c_int32(0)

        def rnd(tm=t, dm=d, prm=p, ws=wb, tcap=128, flags=None):
            tkv.capacity = tcap
            if flags is not None:
                prm = api.RoundParams(prm.k_max, prm.mode, prm.depth, prm.trunk_max,
                                      prm.confidence, prm.temperature, flags)
            return lib.sb_spec_round(tm, C.byref(tkv), 100, dm, C.byref(dkv), 100, C.byref(prm),
                                     1, 1, 1, 1, 1, 1, 1, 1, 1, 1, 1, par, C.byref(nc),
                                     C.byref(nb), 1, ws, None, None)
        assert rnd(dm=None) == 1
        assert rnd(dm=t) == 1                       # the target and the draft are one model
        assert rnd(flags=2) == 1                     # unknown flag
        assert rnd(prm=api.RoundParams(4, 2, 3, 4, float("nan"), 1.0, 0)) == 1
        assert rnd(prm=api.RoundParams(4, 2, 3, 4, 0.1, -1.0, 0)) == 1
        assert rnd(ws=wb - 1) == 3
        assert rnd(tcap=100) == 3                    # no room for the chain's rows
    finally:
        lib.sb_model_destroy(t)
        lib.sb_model_destroy(d)
