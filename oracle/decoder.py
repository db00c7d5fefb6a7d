"""Oracle target forward over a token tree (test infrastructure only).

The paper's target models are Llama-family decoders (Appendix, "Model
Configurations", Table 7); the verification phase of Algorithm 2 scores all
draft positions of a round with one target forward.  This module is the
plain definition of that forward for a token *tree* whose rows share one
prefix KV cache:

  for every row i with token t_i at position pos(i) = P_kv + depth(i):
    h = E[t_i]
    per layer:
      a = RMSNorm(h) * g1
      q, k, v = a Wq^T, a Wk^T, a Wv^T            (no bias)
      q, k = RoPE(q, pos(i)), RoPE(k, pos(i))     (rotate-half pairing,
                                                   theta_j = base^(-2j/d))
      o = softmax(q K_i^T / sqrt(d)) V_i          keys K_i, V_i: the prefix
          slots 0..P_kv-1, then the tree rows on the path root..i (ascending
          depth); query head h reads KV head floor(h * n_kv / n_heads)
      h = h + o Wo^T
      m = RMSNorm(h) * g2
      h = h + (silu(m Wg^T) * (m Wu^T)) Wd^T
    logits = (RMSNorm(h) * g_f) W_lm^T            (untied LM head)

The key order for row i is exactly the order a fresh causal prefill of
prefix + path(i) would use, so each branch's rows equal a plain causal
forward of that branch (the paper keeps the branch that survives and drops
the others, Section "Branch Resampling", "Branch Verification").

Every RMSNorm feeds a projection, and the oracle applies it in the
factored form RMSNorm(h) g W^T = r (h g) W^T with r = 1/sqrt(mean(h^2) + eps)
per row: the projection's input is h g, and its output is multiplied by r.
The two forms are equal in exact arithmetic; the factored one fixes where a
reduced-precision implementation rounds.

Precision modes:
  "f64"      everything in float64;
  "f32"      everything in float32;
  "bf16"     float32 arithmetic with values rounded to bfloat16 (nearest
             even) at exactly these points, where the GPU path stores
             bfloat16 tensors (the bf16 rounding-point contract):
               1. each norm's projection input, bf16(h g);
               2. q and k after RoPE, and v;
               3. the attention output o = p V (the probabilities p are
                  not rounded);
               4. the SwiGLU product silu(gate) up;
               and the KV cache holds the rounded k and v.  The residual
             stream h, the row scales r, the projections' outputs and the
             logits stay float32;
  "bf16_f64" the same rounding points with float64 arithmetic (each rounded
             value passes through float32 first, as a float32 value stored
             as bfloat16 would).
"""
from __future__ import annotations

import math

import numpy as np

from . import tree


def round_bf16(x: np.ndarray) -> np.ndarray:
    """float32 -> nearest-even bfloat16 value, returned as float32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000).astype(np.uint32)
    return r.view(np.float32).reshape(x.shape)


class _Prec:
    def __init__(self, mode: str):
        if mode not in ("f64", "f32", "bf16", "bf16_f64"):
            raise ValueError(mode)
        self.mode = mode
        self.dt = np.float64 if mode in ("f64", "bf16_f64") else np.float32

    def cast(self, x):
        return np.asarray(x, dtype=self.dt)

    def store(self, x):
        """Value as the GPU path stores it (bf16 rounding in the bf16 modes)."""
        x = np.asarray(x, dtype=self.dt)
        if self.mode == "bf16":
            return round_bf16(x)
        if self.mode == "bf16_f64":
            return round_bf16(x.astype(np.float32)).astype(np.float64)
        return x


def rms_norm(x: np.ndarray, g: np.ndarray, eps: float, dt) -> np.ndarray:
    x = x.astype(dt)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return (x / np.sqrt(ms + dt(eps))) * g.astype(dt)


def rms_scale(x: np.ndarray, eps: float, dt) -> np.ndarray:
    """r = 1/sqrt(mean(x^2) + eps) per row, shape [rows][1]."""
    x = x.astype(dt)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return dt(1) / np.sqrt(ms + dt(eps))


def rope_tables(pos: np.ndarray, head_dim: int, base: float, dt):
    """cos/sin of pos * theta_j, theta_j = base^(-2j/d), j < d/2 (float64
    angles, cast to the working precision)."""
    j = np.arange(head_dim // 2, dtype=np.float64)
    theta = np.power(np.float64(base), -2.0 * j / head_dim)
    ang = pos.astype(np.float64)[:, None] * theta[None, :]
    return np.cos(ang).astype(dt), np.sin(ang).astype(dt)


def apply_rope(x: np.ndarray, cos: np.ndarray, sin: np.ndarray) -> np.ndarray:
    """x: [rows][heads][d]; rotate-half pairing of element j with j + d/2."""
    half = x.shape[-1] // 2
    x1, x2 = x[..., :half], x[..., half:]
    c, s = cos[:, None, :], sin[:, None, :]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(x: np.ndarray) -> np.ndarray:
    one = x.dtype.type(1)
    return x / (one + np.exp(-x))


def tree_forward(shape, weights: dict, prefix_k, prefix_v, kv_len: int, tokens, parents,
                 mode: str = "f64", hidden: list | None = None):
    """Forward of the token tree (tokens[i], parents[i]) on a prefix KV cache.

    prefix_k / prefix_v: per layer [n_kv_heads][>= kv_len][head_dim] arrays
    (a list, or an array with a leading layer axis; only slots < kv_len are
    read).  Returns (logits [N][V], k_tree, v_tree) where k_tree / v_tree are
    [n_layers][n_kv_heads][N][head_dim]: the keys/values the tree rows write
    to cache slots kv_len + i.  If `hidden` is a list, the residual stream
    after every layer ([N][hidden], layer 0 first) is appended to it.
    """
    P = _Prec(mode)
    dt = P.dt
    tokens = np.asarray(tokens, dtype=np.int64)
    parents = np.asarray(parents, dtype=np.int64)
    tree.validate(parents)
    N = len(tokens)
    nh, nkv, d = shape.n_heads, shape.n_kv_heads, shape.head_dim
    eps = shape.rms_eps
    pos = kv_len + tree.depths(parents)
    cos, sin = rope_tables(pos, d, shape.rope_theta, dt)
    paths = [tree.root_path(parents, i) for i in range(N)]
    scale = dt(1.0 / math.sqrt(d))

    h = P.cast(weights["embed"][tokens])
    k_tree = np.zeros((shape.n_layers, nkv, N, d), dtype=dt)
    v_tree = np.zeros((shape.n_layers, nkv, N, d), dtype=dt)
    for li in range(shape.n_layers):
        W = weights["layers"][li]
        # RMSNorm(h) g1 W^T = r1 (h g1) W^T
        r1 = rms_scale(h, eps, dt)
        a = P.store(h * P.cast(W["attn_norm"]))
        q = ((a @ P.cast(W["wq"]).T) * r1).reshape(N, nh, d)
        k = ((a @ P.cast(W["wk"]).T) * r1).reshape(N, nkv, d)
        v = ((a @ P.cast(W["wv"]).T) * r1).reshape(N, nkv, d)
        q = P.store(apply_rope(q, cos, sin))
        k = P.store(apply_rope(k, cos, sin))
        v = P.store(v)
        k_tree[li] = k.transpose(1, 0, 2)
        v_tree[li] = v.transpose(1, 0, 2)
        pk = P.cast(np.asarray(prefix_k[li])[:, :kv_len]) if kv_len else np.zeros((nkv, 0, d), dt)
        pv = P.cast(np.asarray(prefix_v[li])[:, :kv_len]) if kv_len else np.zeros((nkv, 0, d), dt)
        o = np.zeros((N, nh, d), dtype=dt)
        for i in range(N):
            rows = paths[i]
            for hh in range(nh):
                g = hh * nkv // nh
                K = np.concatenate([pk[g], k[rows, g]], axis=0)
                V = np.concatenate([pv[g], v[rows, g]], axis=0)
                s = (K @ q[i, hh]) * scale
                e = np.exp(s - s.max())
                p = e / e.sum()
                o[i, hh] = p @ V
        o = P.store(o.reshape(N, nh * d))
        h = h + o @ P.cast(W["wo"]).T
        # RMSNorm(h) g2 W^T = r2 (h g2) W^T for the gate and up projections
        r2 = rms_scale(h, eps, dt)
        m = P.store(h * P.cast(W["mlp_norm"]))
        gt = (m @ P.cast(W["wg"]).T) * r2
        up = (m @ P.cast(W["wu"]).T) * r2
        act = P.store(silu(gt) * up)
        h = h + act @ P.cast(W["wd"]).T
        if hidden is not None:
            hidden.append(h.copy())
    rf = rms_scale(h, eps, dt)
    fin = P.store(h * P.cast(weights["final_norm"]))
    logits = (fin @ P.cast(weights["lm_head"]).T) * rf
    return logits, k_tree, v_tree


def prefill(shape, weights: dict, tokens, mode: str = "f64"):
    """Causal forward of a plain token sequence from an empty cache.

    Returns (logits [n][V], K, V) with K, V [n_layers][n_kv][n][d]."""
    n = len(tokens)
    parents = np.arange(-1, n - 1)
    empty = [None] * shape.n_layers
    return tree_forward(shape, weights, empty, empty, 0, tokens, parents, mode)


def make_cache(shape, prefix_k, prefix_v, kv_len: int, capacity: int, dt=np.float64):
    """KV caches [n_layers][n_kv][capacity][d] holding the prefix in slots
    0..kv_len-1 (zeros elsewhere)."""
    K = np.zeros((shape.n_layers, shape.n_kv_heads, capacity, shape.head_dim), dtype=dt)
    V = np.zeros_like(K)
    if kv_len:
        K[:, :, :kv_len] = np.asarray(prefix_k)[:, :, :kv_len]
        V[:, :, :kv_len] = np.asarray(prefix_v)[:, :, :kv_len]
    return K, V


def write_tree_kv(K, V, kv_len: int, k_tree, v_tree):
    """Store tree row i's K/V in slot kv_len + i (what the verify step does)."""
    N = k_tree.shape[2]
    K = K.copy()
    V = V.copy()
    K[:, :, kv_len:kv_len + N] = k_tree
    V[:, :, kv_len:kv_len + N] = v_tree
    return K, V
