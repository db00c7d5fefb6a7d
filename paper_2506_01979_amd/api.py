"""Thin Python binding of libsb (``include/sb.h``) over ctypes.

Argument marshalling only: every step of the verify path runs in the HIP
kernels behind the C ABI.  PyTorch supplies device memory and the stream.
Importing this module loads ``libsb.so`` from the package directory and
raises if it is missing (build it with ``python -m paper_2506_01979_amd.build``).
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np
import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsb.so")
if not os.path.exists(_LIB_PATH):
    raise ImportError(f"{_LIB_PATH} is missing: run `python -m paper_2506_01979_amd.build`")
lib = C.CDLL(_LIB_PATH)

SB_MAX_ROWS = 256
SB_F32, SB_BF16 = 0, 1
SB_W_QKV, SB_W_O, SB_W_GATE_UP, SB_W_DOWN, SB_W_LM_HEAD = range(5)
SB_FLAG_NONFINITE, SB_FLAG_QZERO, SB_FLAG_ZERO_RESIDUAL = 1, 2, 4

STATUS = {0: "SB_OK", 1: "SB_ERR_INVALID_ARG", 2: "SB_ERR_TREE", 3: "SB_ERR_CAPACITY",
          4: "SB_ERR_DTYPE", 5: "SB_ERR_HIP", 6: "SB_ERR_UNSUPPORTED"}

EXPORTS = ("sb_status_string", "sb_version", "sb_packed_bytes", "sb_pack_weight",
           "sb_model_create", "sb_model_destroy", "sb_workspace_bytes", "sb_verify_forward",
           "sb_softmax_stats", "sb_sample_workspace_bytes", "sb_select_branch",
           "sb_accept_resample", "sb_kv_rollback", "sb_timer_start", "sb_timer_stop",
           "sb_model_set_tap", "sb_hrad_workspace_bytes", "sb_hrad_predict",
           "sb_branch_workspace_bytes", "sb_branch_candidates", "sb_draft_sample",
           "sb_draft_sample_workspace_bytes",
           "sb_draft_round_workspace_bytes", "sb_draft_round", "sb_verify_forward_noalloc",
           "sb_model_set_forward", "sb_draft_chain", "sb_draft_branches", "sb_round_finish",
           "sb_spec_round_workspace_bytes", "sb_spec_round")
SB_FWD_AUTO, SB_FWD_KERNELS, SB_FWD_PERSISTENT = 0, 1, 2

SB_HRAD_H1, SB_HRAD_H2, SB_HRAD_CLASSES = 256, 64, 3
BRANCH_MODES = {"topk": 0, "iid": 1, "wor": 2}
SB_BRANCH_MAX_K, SB_BRANCH_MAX_VOCAB = 16, 1048576
SB_DRAFT_MAX_ROWS = 64

KERNEL_CLASSES = {"qkv": 0, "o": 1, "gate_up": 2, "down": 3, "lm_head": 4, "attn": 5,
                  "attn_merge": 6, "norm": 7, "stats": 8, "persist": 9}


class SBError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        msg = lib.sb_status_string(code).decode()
        super().__init__(f"{where}: {STATUS.get(code, code)} ({msg})")


class ModelConfig(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("hidden", C.c_int32), ("n_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("ffn", C.c_int32),
                ("vocab", C.c_int32), ("rope_theta", C.c_float), ("rms_eps", C.c_float),
                ("dtype", C.c_int32)]


class LayerWeights(C.Structure):
    _fields_ = [("attn_norm", C.c_void_p), ("qkv", C.c_void_p), ("o", C.c_void_p),
                ("mlp_norm", C.c_void_p), ("gate_up", C.c_void_p), ("down", C.c_void_p)]


class ModelWeights(C.Structure):
    _fields_ = [("embed", C.c_void_p), ("final_norm", C.c_void_p), ("lm_head", C.c_void_p),
                ("layers", C.POINTER(LayerWeights))]


class KVCache(C.Structure):
    _fields_ = [("k", C.c_void_p), ("v", C.c_void_p), ("capacity", C.c_int32)]


class HradWeights(C.Structure):
    _fields_ = [("w1", C.c_void_p), ("b1", C.c_void_p), ("w2", C.c_void_p),
                ("b2", C.c_void_p), ("w3", C.c_void_p), ("b3", C.c_void_p)]


SB_CHAIN_CONDITIONED = 1


class RoundParams(C.Structure):
    _fields_ = [("k_max", C.c_int32), ("mode", C.c_int32), ("depth", C.c_int32),
                ("trunk_max", C.c_int32), ("confidence", C.c_float), ("temperature", C.c_float),
                ("flags", C.c_int32)]


ROUND_RESULT_INTS = 8
ROW_STATS_DTYPE = np.dtype([("zmax", "<f4"), ("argmax", "<i4"), ("total", "<f8")])
STEP_RESULT_INTS = 8 + SB_MAX_ROWS

_vp, _i32, _sz, _f = C.c_void_p, C.c_int32, C.c_size_t, C.c_float
lib.sb_status_string.restype = C.c_char_p
lib.sb_status_string.argtypes = [_i32]
lib.sb_version.restype = _i32
lib.sb_packed_bytes.restype = _sz
lib.sb_packed_bytes.argtypes = [C.POINTER(ModelConfig), _i32]
lib.sb_pack_weight.restype = _i32
lib.sb_pack_weight.argtypes = [C.POINTER(ModelConfig), _i32, _vp, _vp, _vp, _vp, _vp]
lib.sb_model_create.restype = _i32
lib.sb_model_create.argtypes = [C.POINTER(ModelConfig), C.POINTER(ModelWeights), C.POINTER(_vp)]
lib.sb_model_destroy.restype = None
lib.sb_model_destroy.argtypes = [_vp]
lib.sb_workspace_bytes.restype = _sz
lib.sb_workspace_bytes.argtypes = [_vp, _i32, _i32]
lib.sb_verify_forward.restype = _i32
lib.sb_verify_forward.argtypes = [_vp, C.POINTER(KVCache), _i32, _vp, C.POINTER(_i32), _i32, _f,
                                  _vp, _vp, _vp, _sz, _vp]
lib.sb_verify_forward_noalloc.restype = _i32
lib.sb_verify_forward_noalloc.argtypes = [_vp, C.POINTER(KVCache), _i32, _vp, C.POINTER(_i32),
                                          _i32, _f, _vp, _vp, _vp]
SB_NOALLOC_SCRATCH_BYTES = 128 * 1024 * 1024
lib.sb_model_set_forward.restype = _i32
lib.sb_model_set_forward.argtypes = [_vp, _i32]
lib.sb_softmax_stats.restype = _i32
lib.sb_softmax_stats.argtypes = [_i32, _i32, _vp, _f, _vp, _vp]
lib.sb_sample_workspace_bytes.restype = _sz
lib.sb_sample_workspace_bytes.argtypes = [_i32]
lib.sb_select_branch.restype = _i32
lib.sb_select_branch.argtypes = [_i32, _vp, _vp, _f, _i32, _vp, _vp, _vp, _vp, _vp, _sz, _vp]
lib.sb_accept_resample.restype = _i32
lib.sb_accept_resample.argtypes = [_i32, _i32, _vp, C.POINTER(_i32), _vp, _vp, _f, _vp, _vp, _vp,
                                   _vp, _sz, _vp]
lib.sb_timer_start.restype = _i32
lib.sb_timer_start.argtypes = [_vp, _i32, _i32]
lib.sb_timer_stop.restype = _i32
lib.sb_timer_stop.argtypes = [_vp, C.POINTER(C.c_double), C.POINTER(_i32)]
lib.sb_kv_rollback.restype = _i32
lib.sb_kv_rollback.argtypes = [_vp, C.POINTER(KVCache), _i32, _vp, _vp, _vp]
lib.sb_model_set_tap.restype = _i32
lib.sb_model_set_tap.argtypes = [_vp, _vp, _i32, _i32]
lib.sb_hrad_workspace_bytes.restype = _sz
lib.sb_hrad_workspace_bytes.argtypes = []
lib.sb_branch_workspace_bytes.restype = _sz
lib.sb_branch_workspace_bytes.argtypes = []
lib.sb_branch_candidates.restype = _i32
lib.sb_branch_candidates.argtypes = [_vp, _i32, _vp, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _sz,
                                     _vp]
lib.sb_draft_sample.restype = _i32
lib.sb_draft_sample.argtypes = [_i32, _i32, _vp, _vp, _i32, C.POINTER(_i32), _f, _vp, _vp, _vp,
                                _i32, C.POINTER(_i32), _vp, _sz, _vp]
lib.sb_draft_sample_workspace_bytes.restype = _sz
lib.sb_draft_sample_workspace_bytes.argtypes = [_i32, _i32]
lib.sb_draft_round_workspace_bytes.restype = _sz
lib.sb_draft_round_workspace_bytes.argtypes = [_vp, _i32, _i32, _i32, _i32]
lib.sb_draft_round.restype = _i32
lib.sb_draft_round.argtypes = [_vp, C.POINTER(KVCache), _i32, _i32, _i32, _i32, _i32, _f, _f, _vp,
                               _vp, _vp, C.POINTER(_i32), C.POINTER(_i32), C.POINTER(_i32), _vp,
                               _sz, _vp]
lib.sb_draft_chain.restype = _i32
lib.sb_draft_chain.argtypes = [_vp, C.POINTER(KVCache), _i32, _i32, _f, _i32, _f, _vp, _vp, _vp,
                               _vp, C.POINTER(_i32), _vp, _sz, _vp]
lib.sb_draft_branches.restype = _i32
lib.sb_draft_branches.argtypes = [_vp, C.POINTER(KVCache), _i32, _i32, _vp, _i32, _i32, _i32, _f,
                                  _vp, _vp, _vp, C.POINTER(_i32), C.POINTER(_i32), _vp, _sz, _vp]
lib.sb_round_finish.restype = _i32
lib.sb_round_finish.argtypes = [_i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp]
lib.sb_spec_round_workspace_bytes.restype = _sz
lib.sb_spec_round_workspace_bytes.argtypes = [_vp, _vp, C.POINTER(RoundParams), _i32, _i32]
lib.sb_spec_round.restype = _i32
lib.sb_spec_round.argtypes = [_vp, C.POINTER(KVCache), _i32, _vp, C.POINTER(KVCache), _i32,
                              C.POINTER(RoundParams), _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                              _vp, _vp, C.POINTER(_i32), C.POINTER(_i32), C.POINTER(_i32), _vp,
                              _sz, _vp, _vp]
lib.sb_hrad_predict.restype = _i32
lib.sb_hrad_predict.argtypes = [_vp, _vp, _i32, _i32, _vp, C.POINTER(HradWeights), _vp, _vp,
                                _vp, _sz, _vp]


def _check(code: int, where: str) -> None:
    if code != 0:
        raise SBError(code, where)


def _need(t: torch.Tensor, nbytes: int, what: str, dtype=None) -> None:
    """Host-side check that a device buffer is large enough before a launch."""
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{what}: expected a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{what}: expected a contiguous tensor")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{what}: expected {dtype}, got {t.dtype}")
    have = t.numel() * t.element_size()
    if have < nbytes:
        raise ValueError(f"{what}: {have} bytes < {nbytes} needed")


def _stream(stream=None) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _ptr(t) -> int | None:
    return None if t is None else t.data_ptr()


def _host_i32(a) -> tuple:
    arr = np.ascontiguousarray(np.asarray(a, dtype=np.int32))
    return arr, arr.ctypes.data_as(C.POINTER(C.c_int32))


def make_config(shape) -> ModelConfig:
    return ModelConfig(shape.n_layers, shape.hidden, shape.n_heads, shape.n_kv_heads,
                       shape.head_dim, shape.ffn, shape.vocab, shape.rope_theta, shape.rms_eps,
                       SB_BF16 if shape.dtype == "bf16" else SB_F32)


# ----------------------------------------------------------------------------
# entry points (same names as the C ABI)
# ----------------------------------------------------------------------------

def sb_packed_bytes(cfg: ModelConfig, kind: int) -> int:
    return int(lib.sb_packed_bytes(C.byref(cfg), kind))


def sb_pack_weight(cfg: ModelConfig, kind: int, srcs, dst: torch.Tensor, stream=None) -> None:
    s = list(srcs) + [None] * (3 - len(srcs))
    _check(lib.sb_pack_weight(C.byref(cfg), kind, _ptr(s[0]), _ptr(s[1]), _ptr(s[2]),
                              dst.data_ptr(), _stream(stream)), "sb_pack_weight")


def sb_softmax_stats(logits: torch.Tensor, temperature: float, stats: torch.Tensor,
                     stream=None) -> None:
    n, v = logits.shape
    _need(logits, n * v * 4, "logits", torch.float32)
    _need(stats, n * 16, "stats")
    _check(lib.sb_softmax_stats(v, n, logits.data_ptr(), temperature, stats.data_ptr(),
                                _stream(stream)), "sb_softmax_stats")


def sb_select_branch(logits_row: torch.Tensor, stats_row: torch.Tensor, temperature: float,
                     cand_tokens: torch.Tensor, q: torch.Tensor, u: torch.Tensor,
                     out: torch.Tensor, ws: torch.Tensor, stream=None) -> None:
    v = logits_row.shape[-1]
    nc = cand_tokens.shape[0]
    _need(logits_row, v * 4, "logits_row", torch.float32)
    _need(stats_row, 16, "stats_row")
    _need(cand_tokens, nc * 4, "cand_tokens", torch.int32)
    _need(q, nc * v * 4, "q", torch.float32)
    _need(u, (nc + 1) * 4, "u", torch.float32)
    _need(out, 12, "out", torch.int32)
    _need(ws, sb_sample_workspace_bytes(v), "ws")
    _check(lib.sb_select_branch(logits_row.shape[-1], logits_row.data_ptr(), stats_row.data_ptr(),
                                temperature, cand_tokens.shape[0], cand_tokens.data_ptr(),
                                q.data_ptr(), u.data_ptr(), out.data_ptr(), ws.data_ptr(),
                                ws.numel() * ws.element_size(), _stream(stream)),
           "sb_select_branch")


def sb_accept_resample(tokens: torch.Tensor, parents, logits: torch.Tensor, stats: torch.Tensor,
                       temperature: float, q: torch.Tensor, u: torch.Tensor,
                       result: torch.Tensor, ws: torch.Tensor, stream=None) -> None:
    n, v = logits.shape[0], logits.shape[1]
    par, pp = _host_i32(parents)
    m = len(par)
    _need(tokens, m * 4, "tokens", torch.int32)
    _need(logits, m * v * 4, "logits", torch.float32)
    _need(stats, m * 16, "stats")
    _need(q, m * v * 4, "q", torch.float32)
    _need(u, m * 4, "u", torch.float32)
    _need(result, STEP_RESULT_INTS * 4, "result", torch.int32)
    _need(ws, sb_sample_workspace_bytes(v), "ws")
    _check(lib.sb_accept_resample(v, len(par), tokens.data_ptr(), pp, logits.data_ptr(),
                                  stats.data_ptr(), temperature, q.data_ptr(), u.data_ptr(),
                                  result.data_ptr(), ws.data_ptr(),
                                  ws.numel() * ws.element_size(), _stream(stream)),
           "sb_accept_resample")


def sb_round_finish(chain: int, branches: int, depth: int, walk: torch.Tensor, select,
                    round_out: torch.Tensor, draft_path: torch.Tensor, stream=None) -> None:
    """walk / draft_path: sb_step_result buffers (new_result()); select int32
    [3] or None when branches = 0; round_out int32 [ROUND_RESULT_INTS]."""
    _need(walk, STEP_RESULT_INTS * 4, "walk", torch.int32)
    if select is not None:
        _need(select, 12, "select", torch.int32)
    _need(round_out, ROUND_RESULT_INTS * 4, "round_out", torch.int32)
    _need(draft_path, STEP_RESULT_INTS * 4, "draft_path", torch.int32)
    _check(lib.sb_round_finish(chain, branches, depth, walk.data_ptr(), _ptr(select),
                               round_out.data_ptr(), draft_path.data_ptr(), _stream(stream)),
           "sb_round_finish")


def new_round_result(device="cuda") -> torch.Tensor:
    return torch.full((ROUND_RESULT_INTS,), -7, dtype=torch.int32, device=device)


def decode_round(r: torch.Tensor) -> dict:
    a = r.cpu().numpy()
    return {"n_trunk": int(a[0]), "kept": int(a[1]), "token": int(a[2]), "flags": int(a[3]),
            "draft_len": int(a[4])}


def round_params(k_max: int, mode: str, depth: int, trunk_max: int, confidence: float,
                 temperature: float, conditioned: bool = False) -> RoundParams:
    return RoundParams(k_max, BRANCH_MODES[mode], depth, trunk_max, confidence, temperature,
                       SB_CHAIN_CONDITIONED if conditioned else 0)


def sb_spec_round_workspace_bytes(target, draft, params: RoundParams, t_len: int,
                                  d_len: int) -> int:
    return int(lib.sb_spec_round_workspace_bytes(target.handle, draft.handle, C.byref(params),
                                                 t_len, d_len))


class RoundBuffers:
    """Device buffers of sb_spec_round for one parameter set."""

    def __init__(self, target, draft, params: RoundParams, t_len: int, d_len: int,
                 device="cuda"):
        V = target.shape.vocab
        R = params.trunk_max + params.k_max * params.depth
        self.params = params
        self.tokens = torch.zeros(R, dtype=torch.int32, device=device)
        self.q = torch.zeros((R, V), dtype=torch.float32, device=device)
        self.logits = torch.zeros((params.trunk_max, V), dtype=torch.float32, device=device)
        self.stats = new_stats(params.trunk_max, device)
        self.walk = new_result(device)
        self.select = torch.full((3,), -7, dtype=torch.int32, device=device)
        self.round = new_round_result(device)
        self.new_lens = torch.zeros(2, dtype=torch.int32, device=device)
        n = sb_spec_round_workspace_bytes(target, draft, params, t_len, d_len)
        if n == 0:
            raise ValueError("sb_spec_round_workspace_bytes: arguments rejected")
        self.ws = torch.empty(n, dtype=torch.uint8, device=device)
        self.parents = np.zeros(R, dtype=np.int32)


def sb_spec_round(target, t_k: torch.Tensor, t_v: torch.Tensor, t_len: int, draft,
                  d_k: torch.Tensor, d_v: torch.Tensor, d_len: int, u_draft: torch.Tensor,
                  u_walk: torch.Tensor, u_sel: torch.Tensor, buf: RoundBuffers,
                  verify_stream=None, draft_stream=None):
    """One round (buf.tokens[0] = the root on entry).  Returns (c, B,
    parents of the draft tree).  Both streams default to the current one."""
    p = buf.params
    target._check_kv(t_k, t_v)
    draft._check_kv(d_k, d_v)
    R = p.trunk_max + p.k_max * p.depth
    _need(u_draft, R * 4, "u_draft", torch.float32)
    _need(u_walk, (p.trunk_max + 1) * 4, "u_walk", torch.float32)
    _need(u_sel, (p.k_max + 1) * 4, "u_sel", torch.float32)
    tkv = KVCache(t_k.data_ptr(), t_v.data_ptr(), t_k.shape[2])
    dkv = KVCache(d_k.data_ptr(), d_v.data_ptr(), d_k.shape[2])
    nc, nb = C.c_int32(0), C.c_int32(0)
    par = buf.parents
    _check(lib.sb_spec_round(target.handle, C.byref(tkv), t_len, draft.handle, C.byref(dkv), d_len,
                             C.byref(p), u_draft.data_ptr(), u_walk.data_ptr(), u_sel.data_ptr(),
                             buf.tokens.data_ptr(), buf.q.data_ptr(), buf.logits.data_ptr(),
                             buf.stats.data_ptr(), buf.walk.data_ptr(), buf.select.data_ptr(),
                             buf.round.data_ptr(), buf.new_lens.data_ptr(),
                             par.ctypes.data_as(C.POINTER(C.c_int32)), C.byref(nc), C.byref(nb),
                             buf.ws.data_ptr(), buf.ws.numel(), _stream(verify_stream),
                             _stream(draft_stream)), "sb_spec_round")
    c, B = int(nc.value), int(nb.value)
    return c, B, par[:1 + c + B * p.depth].copy()


def sb_branch_workspace_bytes() -> int:
    return int(lib.sb_branch_workspace_bytes())


def sb_branch_candidates(q: torch.Tensor, x_b: torch.Tensor, k_max: int, mode: str, u,
                         count: torch.Tensor, tokens: torch.Tensor, rows: torch.Tensor,
                         ws: torch.Tensor, stream=None) -> None:
    """q float32 [vocab]; x_b int32 [1] on the device; u float32 [k_max] (None
    for "topk"); count int32 [1]; tokens int32 [k_max]; rows float32
    [k_max][vocab]."""
    v = q.shape[-1]
    _need(q, v * 4, "q", torch.float32)
    _need(x_b, 4, "x_b", torch.int32)
    if u is not None:
        _need(u, k_max * 4, "u", torch.float32)
    _need(count, 4, "count", torch.int32)
    _need(tokens, k_max * 4, "tokens", torch.int32)
    _need(rows, k_max * v * 4, "rows", torch.float32)
    _need(ws, sb_branch_workspace_bytes(), "ws")
    _check(lib.sb_branch_candidates(q.data_ptr(), v, x_b.data_ptr(), k_max, BRANCH_MODES[mode], _ptr(u),
                                    count.data_ptr(), tokens.data_ptr(), rows.data_ptr(),
                                    ws.data_ptr(), ws.numel() * ws.element_size(),
                                    _stream(stream)), "sb_branch_candidates")


def sb_draft_sample_workspace_bytes(vocab: int, n: int) -> int:
    return int(lib.sb_draft_sample_workspace_bytes(vocab, n))


def sb_draft_sample(logits: torch.Tensor, stats: torch.Tensor, src_rows, temperature: float,
                    u: torch.Tensor, tokens: torch.Tensor, q: torch.Tensor, dst_rows,
                    ws: torch.Tensor, stream=None) -> None:
    """logits float32 [n_logit_rows][vocab] with stats; tokens int32 [n_out];
    q float32 [n_out][vocab]; u float32 [len(src_rows)]."""
    nl, v = logits.shape
    src, sp = _host_i32(src_rows)
    dst, dp = _host_i32(dst_rows)
    if len(src) != len(dst):
        raise ValueError("src_rows and dst_rows differ in length")
    n_out = tokens.numel()
    _need(logits, nl * v * 4, "logits", torch.float32)
    _need(stats, nl * 16, "stats")
    _need(u, len(src) * 4, "u", torch.float32)
    _need(tokens, n_out * 4, "tokens", torch.int32)
    _need(q, n_out * v * 4, "q", torch.float32)
    _need(ws, sb_draft_sample_workspace_bytes(v, len(src)), "ws")
    _check(lib.sb_draft_sample(v, len(src), logits.data_ptr(), stats.data_ptr(), nl, sp,
                               temperature, u.data_ptr(), tokens.data_ptr(), q.data_ptr(), n_out,
                               dp, ws.data_ptr(), ws.numel() * ws.element_size(), _stream(stream)),
           "sb_draft_sample")


def sb_sample_workspace_bytes(vocab: int) -> int:
    return int(lib.sb_sample_workspace_bytes(vocab))


def new_stats(n: int, device="cuda") -> torch.Tensor:
    return torch.empty((n, 4), dtype=torch.int32, device=device)


def new_result(device="cuda") -> torch.Tensor:
    return torch.full((STEP_RESULT_INTS,), -7, dtype=torch.int32, device=device)


def decode_stats(stats: torch.Tensor) -> np.ndarray:
    return stats.cpu().numpy().view(ROW_STATS_DTYPE).reshape(-1)


def decode_result(res: torch.Tensor) -> dict:
    a = res.cpu().numpy()
    plen = int(a[3])
    return {"n_accepted": int(a[0]), "branch": int(a[1]), "next_token": int(a[2]),
            "path_len": plen, "flags": int(a[4]), "n_rejected": int(a[5]), "bonus": int(a[6]),
            "path": [int(x) for x in a[8:8 + max(0, min(plen, SB_MAX_ROWS))]]}


def synth_tensors(shape, seed: int = 0, bits: bool = True):
    """tensor_fn over the seeded synthetic weights (bf16 shapes as bit
    patterns, so the upload moves 2 bytes per weight)."""
    from . import synth

    def fn(name, layer=None):
        if name.endswith("norm"):
            return synth.norm_gain(shape)
        return synth.weight(shape, name, layer, seed, as_bits=bits and shape.dtype == "bf16")
    return fn


def dict_tensors(weights: dict):
    """tensor_fn over a weights dict shaped like ``synth.model_weights``."""
    def fn(name, layer=None):
        if layer is None:
            return weights[name]
        return weights["layers"][layer][name]
    return fn


class Model:
    """A model handle with its packed weights resident on the device.

    ``tensor_fn(name, layer)`` returns one weight as a numpy array (float32,
    or uint16 bfloat16 bit patterns); names are ``embed``, ``lm_head``,
    ``final_norm`` and per layer ``wq wk wv wo wg wu wd attn_norm mlp_norm``.
    Tensors are uploaded one at a time and packed with ``sb_pack_weight``;
    the unpacked sources are freed once packed.
    """

    def __init__(self, shape, tensor_fn, device="cuda", stream=None):
        self.shape = shape
        self.cfg = make_config(shape)
        self.device = device
        self.bf16 = shape.dtype == "bf16"
        self.wdtype = torch.bfloat16 if self.bf16 else torch.float32
        self._keep = []
        st = stream if stream is not None else torch.cuda.current_stream()

        def up(name, layer=None):
            a = np.ascontiguousarray(tensor_fn(name, layer))
            if a.dtype == np.uint16:   # bfloat16 bit patterns
                t = torch.from_numpy(a.view(np.int16)).to(device).view(torch.bfloat16)
            else:
                t = torch.from_numpy(a).to(device=device, dtype=self.wdtype)
            return t.to(self.wdtype)

        def norm(name, layer=None):
            t = torch.from_numpy(np.ascontiguousarray(tensor_fn(name, layer), dtype=np.float32))
            t = t.to(device)
            self._keep.append(t)
            return t

        def pack(kind, names, layer=None):
            srcs = [up(n, layer) for n in names]
            dst = torch.empty(sb_packed_bytes(self.cfg, kind), dtype=torch.uint8, device=device)
            sb_pack_weight(self.cfg, kind, srcs, dst, st)
            st.synchronize()
            del srcs
            self._keep.append(dst)
            return dst

        self.embed = up("embed")
        self._keep.append(self.embed)
        fin = norm("final_norm")
        self.lm_head = pack(SB_W_LM_HEAD, ["lm_head"])
        layers = (LayerWeights * shape.n_layers)()
        for l in range(shape.n_layers):
            qkv = pack(SB_W_QKV, ["wq", "wk", "wv"], l)
            o = pack(SB_W_O, ["wo"], l)
            gu = pack(SB_W_GATE_UP, ["wg", "wu"], l)
            dn = pack(SB_W_DOWN, ["wd"], l)
            layers[l] = LayerWeights(norm("attn_norm", l).data_ptr(), qkv.data_ptr(),
                                     o.data_ptr(), norm("mlp_norm", l).data_ptr(),
                                     gu.data_ptr(), dn.data_ptr())
        self._layers = layers
        mw = ModelWeights(self.embed.data_ptr(), fin.data_ptr(), self.lm_head.data_ptr(), layers)
        h = C.c_void_p()
        _check(lib.sb_model_create(C.byref(self.cfg), C.byref(mw), C.byref(h)), "sb_model_create")
        self.handle = h
        # bound now: at interpreter exit the module's globals may be gone
        # before the model is collected
        self._destroy = lib.sb_model_destroy

    def __del__(self):
        if getattr(self, "handle", None) and getattr(self, "_destroy", None):
            self._destroy(self.handle)
            self.handle = None

    def _check_kv(self, k: torch.Tensor, v: torch.Tensor) -> None:
        s = self.shape
        if k.dim() != 4 or tuple(k.shape[:2]) != (s.n_layers, s.n_kv_heads) \
                or k.shape[3] != s.head_dim:
            raise ValueError("k cache must be [n_layers][n_kv][capacity][head_dim]")
        if v.dim() != 4 or tuple(v.shape) != (s.n_layers, s.n_kv_heads, s.head_dim, k.shape[2]):
            raise ValueError("v cache must be [n_layers][n_kv][head_dim][capacity]")
        if k.shape[2] % 8:
            raise ValueError("cache capacity must be a multiple of 8")
        for t, nm in ((k, "k"), (v, "v")):
            _need(t, t.numel() * t.element_size(), nm, self.wdtype)

    def new_kv(self, capacity: int):
        """Zeroed caches: K [n_layers][n_kv][capacity][head_dim] and V stored
        transposed, [n_layers][n_kv][head_dim][capacity] (capacity is rounded
        up to a multiple of 8)."""
        s = self.shape
        capacity = (capacity + 7) // 8 * 8
        k = torch.zeros((s.n_layers, s.n_kv_heads, capacity, s.head_dim), dtype=self.wdtype,
                        device=self.device)
        v = torch.zeros((s.n_layers, s.n_kv_heads, s.head_dim, capacity), dtype=self.wdtype,
                        device=self.device)
        return k, v

    def load_kv(self, k: torch.Tensor, v: torch.Tensor, K, V, n: int, start: int = 0) -> None:
        """Writes host K/V rows given as [n_layers][n_kv][n][head_dim] (float32
        values or bf16 bit patterns) into slots start..start+n-1."""
        def dev(a):
            a = np.ascontiguousarray(a)
            if a.dtype == np.uint16:
                return torch.from_numpy(a.view(np.int16)).to(self.device).view(torch.bfloat16)
            return torch.from_numpy(np.asarray(a, np.float32)).to(self.device).to(self.wdtype)
        k[:, :, start:start + n] = dev(np.asarray(K)[:, :, :n])
        v[:, :, :, start:start + n] = dev(np.asarray(V)[:, :, :n]).transpose(2, 3)

    @staticmethod
    def read_kv(k: torch.Tensor, v: torch.Tensor, start: int, n: int):
        """Slots start..start+n-1 as float32 arrays [n_layers][n_kv][n][head_dim]."""
        K = k[:, :, start:start + n].float().cpu().numpy()
        V = v[:, :, :, start:start + n].float().transpose(2, 3).cpu().numpy()
        return K, V

    def workspace(self, max_rows: int, max_kv_len: int) -> torch.Tensor:
        n = int(lib.sb_workspace_bytes(self.handle, max_rows, max_kv_len))
        if n == 0:
            raise SBError(1, "sb_workspace_bytes")
        return torch.empty(n, dtype=torch.uint8, device=self.device)

    def sb_verify_forward(self, k: torch.Tensor, v: torch.Tensor, kv_len: int,
                          tokens: torch.Tensor, parents, temperature: float,
                          logits: torch.Tensor, stats: torch.Tensor, ws: torch.Tensor,
                          stream=None) -> None:
        self._check_kv(k, v)
        kv = KVCache(k.data_ptr(), v.data_ptr(), k.shape[2])
        par, pp = _host_i32(parents)
        n = len(par)
        _need(tokens, n * 4, "tokens", torch.int32)
        _need(logits, n * self.shape.vocab * 4, "logits", torch.float32)
        _need(stats, n * 16, "stats")
        _check(lib.sb_verify_forward(self.handle, C.byref(kv), kv_len, tokens.data_ptr(), pp,
                                     len(par), temperature, logits.data_ptr(), stats.data_ptr(),
                                     ws.data_ptr(), ws.numel() * ws.element_size(),
                                     _stream(stream)), "sb_verify_forward")

    def sb_verify_forward_noalloc(self, k: torch.Tensor, v: torch.Tensor, kv_len: int,
                                  tokens: torch.Tensor, parents, temperature: float,
                                  logits: torch.Tensor, stats: torch.Tensor, stream=None) -> None:
        self._check_kv(k, v)
        kv = KVCache(k.data_ptr(), v.data_ptr(), k.shape[2])
        par, pp = _host_i32(parents)
        n = len(par)
        _need(tokens, n * 4, "tokens", torch.int32)
        _need(logits, n * self.shape.vocab * 4, "logits", torch.float32)
        _need(stats, n * 16, "stats")
        _check(lib.sb_verify_forward_noalloc(self.handle, C.byref(kv), kv_len, tokens.data_ptr(),
                                             pp, len(par), temperature, logits.data_ptr(),
                                             stats.data_ptr(), _stream(stream)),
               "sb_verify_forward_noalloc")

    def sb_timer_start(self, kernel_class: str, capacity: int) -> None:
        _check(lib.sb_timer_start(self.handle, KERNEL_CLASSES[kernel_class], capacity),
               "sb_timer_start")

    def sb_timer_stop(self) -> tuple[float, int]:
        ms = C.c_double()
        n = C.c_int32()
        _check(lib.sb_timer_stop(self.handle, C.byref(ms), C.byref(n)), "sb_timer_stop")
        return ms.value, n.value

    def sb_model_set_forward(self, mode: int) -> None:
        _check(lib.sb_model_set_forward(self.handle, mode), "sb_model_set_forward")

    def sb_model_set_tap(self, taps, k_layers: int = 0, max_rows: int = 0) -> None:
        """H-RAD feature tap: later forwards write the residual after each of
        the last k_layers layers to taps, float32 [k_layers][max_rows][hidden]
        (None clears it; the tensor must outlive its use)."""
        if taps is None:
            _check(lib.sb_model_set_tap(self.handle, None, 0, 0), "sb_model_set_tap")
            self._tap = None
            return
        _need(taps, k_layers * max_rows * self.shape.hidden * 4, "taps", torch.float32)
        _check(lib.sb_model_set_tap(self.handle, taps.data_ptr(), k_layers, max_rows),
               "sb_model_set_tap")
        self._tap = taps

    def sb_hrad_predict(self, taps: torch.Tensor, k_layers: int, max_rows: int,
                        result: torch.Tensor, w: dict, logits3: torch.Tensor,
                        cls: torch.Tensor, ws: torch.Tensor, stream=None) -> None:
        """H-RAD's class for the next round from the taps at the walk's last
        accepted row and the embedding of its next token; w: float32 device
        tensors w1 [256][(k+1)*hidden], b1, w2 [64][256], b2, w3 [3][64], b3."""
        H = self.shape.hidden
        _need(taps, k_layers * max_rows * H * 4, "taps", torch.float32)
        _need(result, STEP_RESULT_INTS * 4, "result", torch.int32)
        shapes = {"w1": SB_HRAD_H1 * (k_layers + 1) * H, "b1": SB_HRAD_H1,
                  "w2": SB_HRAD_H2 * SB_HRAD_H1, "b2": SB_HRAD_H2,
                  "w3": SB_HRAD_CLASSES * SB_HRAD_H2, "b3": SB_HRAD_CLASSES}
        for nm, cnt in shapes.items():
            _need(w[nm], cnt * 4, nm, torch.float32)
        _need(logits3, SB_HRAD_CLASSES * 4, "logits3", torch.float32)
        _need(cls, 4, "cls", torch.int32)
        _need(ws, int(lib.sb_hrad_workspace_bytes()), "ws")
        hw = HradWeights(*(w[nm].data_ptr() for nm in ("w1", "b1", "w2", "b2", "w3", "b3")))
        _check(lib.sb_hrad_predict(self.handle, taps.data_ptr(), k_layers, max_rows,
                                   result.data_ptr(), C.byref(hw), logits3.data_ptr(),
                                   cls.data_ptr(), ws.data_ptr(), ws.numel() * ws.element_size(),
                                   _stream(stream)), "sb_hrad_predict")

    def draft_round_workspace(self, k_max: int, depth: int, kv_len: int,
                              trunk_max: int = 1) -> torch.Tensor:
        n = int(lib.sb_draft_round_workspace_bytes(self.handle, k_max, depth, trunk_max, kv_len))
        if n == 0:
            raise ValueError("sb_draft_round_workspace_bytes: arguments rejected")
        return torch.empty(n, dtype=torch.uint8, device=self.device)

    def sb_draft_round(self, k: torch.Tensor, v: torch.Tensor, kv_len: int, k_max: int, mode: str,
                       depth: int, temperature: float, u: torch.Tensor, tokens: torch.Tensor,
                       q: torch.Tensor, ws: torch.Tensor, stream=None, trunk_max: int = 1,
                       confidence: float = float("inf")):
        """tokens int32 [trunk_max + k_max*depth] with tokens[0] the root on
        entry; q float32 [same][vocab]; u float32 [same].  Returns (B,
        parents as a numpy int32 array of 1 + c + B*depth entries, c)."""
        self._check_kv(k, v)
        R = trunk_max + k_max * depth
        V = self.shape.vocab
        _need(u, R * 4, "u", torch.float32)
        _need(tokens, R * 4, "tokens", torch.int32)
        _need(q, R * V * 4, "q", torch.float32)
        par = np.zeros(R, dtype=np.int32)
        nb, nc = C.c_int32(0), C.c_int32(0)
        kv = KVCache(k.data_ptr(), v.data_ptr(), k.shape[2])
        _check(lib.sb_draft_round(self.handle, C.byref(kv), kv_len, k_max, BRANCH_MODES[mode],
                                  depth, trunk_max, confidence, temperature, u.data_ptr(),
                                  tokens.data_ptr(), q.data_ptr(),
                                  par.ctypes.data_as(C.POINTER(C.c_int32)), C.byref(nb),
                                  C.byref(nc), ws.data_ptr(), ws.numel() * ws.element_size(),
                                  _stream(stream)), "sb_draft_round")
        B, c = int(nb.value), int(nc.value)
        return B, par[:1 + c + B * depth].copy(), c

    def sb_draft_chain(self, k: torch.Tensor, v: torch.Tensor, kv_len: int, trunk_max: int,
                       confidence: float, temperature: float, u: torch.Tensor,
                       tokens: torch.Tensor, q: torch.Tensor, xb: torch.Tensor, ws: torch.Tensor,
                       stream=None, conditioned: bool = False) -> int:
        """tokens int32 / q float32 [>= trunk_max + 1]([vocab]), tokens[0] the
        root; u float32 [trunk_max]; xb int32 [1]; ws of
        draft_round_workspace(1, 1, kv_len, trunk_max).  Returns c."""
        self._check_kv(k, v)
        V = self.shape.vocab
        _need(u, trunk_max * 4, "u", torch.float32)
        _need(tokens, (trunk_max + 1) * 4, "tokens", torch.int32)
        _need(q, (trunk_max + 1) * V * 4, "q", torch.float32)
        _need(xb, 4, "xb", torch.int32)
        nc = C.c_int32(0)
        kv = KVCache(k.data_ptr(), v.data_ptr(), k.shape[2])
        _check(lib.sb_draft_chain(self.handle, C.byref(kv), kv_len, trunk_max, confidence,
                                  SB_CHAIN_CONDITIONED if conditioned else 0,
                                  temperature, u.data_ptr(), tokens.data_ptr(), q.data_ptr(),
                                  xb.data_ptr(), C.byref(nc), ws.data_ptr(),
                                  ws.numel() * ws.element_size(), _stream(stream)),
               "sb_draft_chain")
        return int(nc.value)

    def sb_draft_branches(self, k: torch.Tensor, v: torch.Tensor, kv_len: int, chain: int,
                          xb: torch.Tensor, k_max: int, mode: str, depth: int,
                          temperature: float, u: torch.Tensor, tokens: torch.Tensor,
                          q: torch.Tensor, ws: torch.Tensor, stream=None):
        """After sb_draft_chain: u float32 [k_max * depth]; tokens / q hold
        at least 1 + chain + k_max * depth rows; ws of
        draft_round_workspace(k_max, depth, kv_len, chain + 1).  Returns (B,
        parents)."""
        self._check_kv(k, v)
        V = self.shape.vocab
        R = 1 + chain + k_max * depth
        _need(u, k_max * depth * 4, "u", torch.float32)
        _need(tokens, R * 4, "tokens", torch.int32)
        _need(q, R * V * 4, "q", torch.float32)
        _need(xb, 4, "xb", torch.int32)
        par = np.zeros(R, dtype=np.int32)
        nb = C.c_int32(0)
        kv = KVCache(k.data_ptr(), v.data_ptr(), k.shape[2])
        _check(lib.sb_draft_branches(self.handle, C.byref(kv), kv_len, chain, xb.data_ptr(), k_max,
                                     BRANCH_MODES[mode], depth, temperature, u.data_ptr(),
                                     tokens.data_ptr(), q.data_ptr(),
                                     par.ctypes.data_as(C.POINTER(C.c_int32)), C.byref(nb),
                                     ws.data_ptr(), ws.numel() * ws.element_size(),
                                     _stream(stream)), "sb_draft_branches")
        B = int(nb.value)
        return B, par[:1 + chain + B * depth].copy()

    def sb_kv_rollback(self, k: torch.Tensor, v: torch.Tensor, kv_len: int,
                       result: torch.Tensor, new_len: torch.Tensor, stream=None) -> None:
        self._check_kv(k, v)
        _need(result, STEP_RESULT_INTS * 4, "result", torch.int32)
        _need(new_len, 4, "new_len", torch.int32)
        kv = KVCache(k.data_ptr(), v.data_ptr(), k.shape[2])
        _check(lib.sb_kv_rollback(self.handle, C.byref(kv), kv_len, result.data_ptr(),
                                  new_len.data_ptr(), _stream(stream)), "sb_kv_rollback")
