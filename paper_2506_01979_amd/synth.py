"""Seeded synthetic inputs for the branch-verification step.

This module is shared by the tests, the benchmark and the oracle's callers.
It holds no arithmetic of the method itself: it only draws weights, prefix
tokens, draft distributions q, draft tokens and the uniforms that the
accept/resample walk consumes, and it defines the model shapes.

Model shapes follow the paper's Table 7 (Llama-family targets: layers, hidden
width, FFN width, vocabulary).  The paper's datasets and trained weights are
not used; every input is drawn from fixed seeds:

* weights: N(0, 0.02) per matrix, numpy PCG64 seeded with
  ``SeedSequence([seed, tensor_index, chunk])`` for chunks of 2**22 elements
  (so a tensor or a single layer can be drawn on its own and in parallel),
  rounded to bfloat16 with round-to-nearest-even for bf16 shapes; RMSNorm
  gains are 1;
* prefix tokens, draft q logits and draft tokens: PCG64 streams from seed 2;
* uniforms: ``numpy.random.Generator(numpy.random.Philox(1)).random(n,
  float32)`` (Philox4x32-10, Salmon et al. 2011), one value per tree row:
  ``u[i]`` is the uniform of draft row ``i`` and ``u[0]`` the final draw.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, replace

import numpy as np

CHUNK = 1 << 22
WEIGHT_STD = 0.02


@dataclass(frozen=True)
class Shape:
    """Llama-style decoder shape (Table 7 of the paper gives the widths)."""

    name: str
    n_layers: int
    hidden: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    vocab: int
    dtype: str = "f32"          # "f32" or "bf16"
    rope_theta: float = 10000.0
    rms_eps: float = 1e-5

    def with_layers(self, n_layers: int) -> "Shape":
        return replace(self, n_layers=n_layers, name=f"{self.name}[{n_layers}L]")

    @property
    def q_dim(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim


@dataclass(frozen=True)
class Workload:
    """One verify step: a shape, a prefix length P and a B x k branch tree."""

    name: str
    shape: Shape
    prefix: int                 # committed prefix length P; KV holds P-1 rows
    branches: int               # B
    depth: int                  # k draft tokens per branch
    q_temp: float               # draft logits are N(0,1)/q_temp
    temperature: float = 1.0    # target sampling temperature T
    kv_from_prefill: bool = True  # False: prefix KV is seeded N(0,1) values

    @property
    def n_rows(self) -> int:
        return 1 + self.branches * self.depth

    @property
    def kv_len(self) -> int:
        return self.prefix - 1


SHAPES = {
    "tiny": Shape("tiny", 2, 256, 4, 4, 64, 688, 1024, "f32"),
    "exact": Shape("exact", 1, 64, 2, 2, 32, 172, 16, "f32"),
    # a four-token vocabulary, small enough to enumerate a whole round's
    # outcomes exactly
    "enum": Shape("enum", 1, 32, 2, 2, 16, 64, 4, "f32"),
    "llama7b": Shape("llama7b", 32, 4096, 32, 32, 128, 11008, 32000, "bf16"),
    "llama13b": Shape("llama13b", 40, 5120, 40, 40, 128, 13824, 32000, "bf16"),
    "llama70b": Shape("llama70b", 80, 8192, 64, 8, 128, 28672, 128256, "bf16"),
    # small bf16 shapes for parity: several tiles per GEMM, ragged K (688),
    # ragged vocabulary (1000) and a grouped-query variant
    "small_bf16": Shape("small_bf16", 2, 256, 4, 4, 64, 688, 1000, "bf16"),
    "small_gqa_bf16": Shape("small_gqa_bf16", 2, 512, 8, 2, 64, 1376, 1000, "bf16"),
    "small_h128_bf16": Shape("small_h128_bf16", 2, 512, 4, 4, 128, 1024, 2048, "bf16"),
    # ragged everywhere: hidden 328 (not a multiple of 16 or 256; != heads x
    # head_dim), ffn 600, vocabulary 1001 (odd)
    "ragged_bf16": Shape("ragged_bf16", 2, 328, 4, 2, 64, 600, 1001, "bf16"),
    # 32 KV heads on a narrow model: few key ranges per head
    "heads32_bf16": Shape("heads32_bf16", 2, 256, 32, 32, 64, 512, 1000, "bf16"),
    # head_dim 128 with grouped queries (two query heads per KV head)
    "gqa128_bf16": Shape("gqa128_bf16", 2, 512, 4, 2, 128, 1024, 1000, "bf16"),
    # grouped queries at head width 128 (8 query heads per KV head, like the
    # 70B shape) on a narrow model
    "small_gqa128_bf16": Shape("small_gqa128_bf16", 2, 1024, 16, 2, 128, 2752, 2000, "bf16"),
    # the paper's 68M draft model: 2 layers, hidden 768, 12 heads x 64, FFN 3072
    "draft68m": Shape("draft68m", 2, 768, 12, 12, 64, 3072, 32000, "bf16"),
}

WORKLOADS = {
    "tiny": Workload("tiny", SHAPES["tiny"], 128, 2, 4, 0.8),
    "exact": Workload("exact", SHAPES["exact"], 8, 3, 3, 1.0),
    "llama7b_b4k8_p2048": Workload("llama7b_b4k8_p2048", SHAPES["llama7b"], 2048, 4, 8, 0.7,
                                   kv_from_prefill=False),
    "llama13b_b4k8_p512": Workload("llama13b_b4k8_p512", SHAPES["llama13b"], 512, 4, 8, 0.7,
                                   kv_from_prefill=False),
    "llama13b_b4k8_p4096": Workload("llama13b_b4k8_p4096", SHAPES["llama13b"], 4096, 4, 8, 0.7,
                                    kv_from_prefill=False),
    "llama13b_b4k8_p8192": Workload("llama13b_b4k8_p8192", SHAPES["llama13b"], 8192, 4, 8, 0.7,
                                    kv_from_prefill=False),
    "llama13b_b8k16_p8192": Workload("llama13b_b8k16_p8192", SHAPES["llama13b"], 8192, 8, 16, 0.7,
                                     kv_from_prefill=False),
    "llama13b_b8k8_p8192": Workload("llama13b_b8k8_p8192", SHAPES["llama13b"], 8192, 8, 8, 0.7,
                                    kv_from_prefill=False),
    "llama70b_b4k8_p4096": Workload("llama70b_b4k8_p4096", SHAPES["llama70b"], 4096, 4, 8, 0.7,
                                    kv_from_prefill=False),
}


# ----------------------------------------------------------------------------
# weights
# ----------------------------------------------------------------------------

LAYER_MATS = ("wq", "wk", "wv", "wo", "wg", "wu", "wd")


def tensor_index(name: str, layer: int | None = None) -> int:
    """Stable index of a weight tensor, used in its seed."""
    if name == "embed":
        return 0
    if name == "lm_head":
        return 1
    return 2 + 7 * int(layer) + LAYER_MATS.index(name)


def tensor_shape(shape: Shape, name: str) -> tuple[int, int]:
    H, F = shape.hidden, shape.ffn
    return {
        "embed": (shape.vocab, H),
        "lm_head": (shape.vocab, H),
        "wq": (shape.q_dim, H),
        "wk": (shape.kv_dim, H),
        "wv": (shape.kv_dim, H),
        "wo": (H, shape.q_dim),
        "wg": (F, H),
        "wu": (F, H),
        "wd": (H, F),
    }[name]


def _workers() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _normal_chunks(seed_words: list[int], n: int, out: np.ndarray) -> None:
    def fill(c: int) -> None:
        lo = c * CHUNK
        hi = min(n, lo + CHUNK)
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed_words + [c])))
        g.standard_normal(hi - lo, dtype=np.float32, out=out[lo:hi])

    nchunks = (n + CHUNK - 1) // CHUNK
    if nchunks == 1:
        fill(0)
    else:
        with ThreadPoolExecutor(_workers()) as ex:
            list(ex.map(fill, range(nchunks)))


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), round to nearest even."""
    import torch  # torch's float->bfloat16 cast rounds to nearest even

    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32)


def weight(shape: Shape, name: str, layer: int | None = None, seed: int = 0,
           as_bits: bool = False) -> np.ndarray:
    """One weight matrix, N(0, 0.02), bf16-rounded for bf16 shapes.

    Returns float32 values (bf16-representable for bf16 shapes), or the
    uint16 bf16 bit patterns when ``as_bits`` is set (bf16 shapes only).
    """
    rows, cols = tensor_shape(shape, name)
    n = rows * cols
    buf = np.empty(n, dtype=np.float32)
    _normal_chunks([seed, tensor_index(name, layer)], n, buf)
    buf *= np.float32(WEIGHT_STD)
    if shape.dtype == "bf16":
        bits = bf16_bits(buf).reshape(rows, cols)
        if as_bits:
            return bits
        return bits_to_f32(bits)
    if as_bits:
        raise ValueError("as_bits needs a bf16 shape")
    return buf.reshape(rows, cols)


def norm_gain(shape: Shape) -> np.ndarray:
    return np.ones(shape.hidden, dtype=np.float32)


def layer_weights(shape: Shape, layer: int, seed: int = 0) -> dict:
    d = {m: weight(shape, m, layer, seed) for m in LAYER_MATS}
    d["attn_norm"] = norm_gain(shape)
    d["mlp_norm"] = norm_gain(shape)
    return d


def model_weights(shape: Shape, seed: int = 0) -> dict:
    """All weights of a (small) model as float32 arrays."""
    return {
        "embed": weight(shape, "embed", None, seed),
        "lm_head": weight(shape, "lm_head", None, seed),
        "final_norm": norm_gain(shape),
        "layers": [layer_weights(shape, l, seed) for l in range(shape.n_layers)],
    }


# ----------------------------------------------------------------------------
# tree, tokens, q, uniforms
# ----------------------------------------------------------------------------

def branch_parents(branches: int, depth: int) -> np.ndarray:
    """Parents of a B x k branch tree: row 0 is the root (last committed
    token); branch b occupies rows 1+b*k .. b*k+k, its first row hangs off
    the root and every later row off the row before it."""
    par = [-1]
    for b in range(branches):
        for j in range(depth):
            par.append(0 if j == 0 else 1 + b * depth + j - 1)
    return np.asarray(par, dtype=np.int32)


def chain_parents(n: int) -> np.ndarray:
    return np.arange(-1, n - 1, dtype=np.int32)


def fork_parents(trunk: int, branches: int, depth: int) -> np.ndarray:
    """Parents of a chain-plus-fork tree, the verification shape of the
    paper's Section "Branch Verification": rows 1..trunk form a chain from
    the root (the drafts before the branch point), and `branches` branches
    of `depth` rows hang off the last of them (the branch point's candidates,
    each followed by its continuation).  trunk = 0 gives branch_parents."""
    par = [-1] + list(range(trunk))
    fork = trunk
    for b in range(branches):
        base = 1 + trunk + b * depth
        for j in range(depth):
            par.append(fork if j == 0 else base + j - 1)
    return np.asarray(par, dtype=np.int32)


def tree_depths(parents: np.ndarray) -> np.ndarray:
    """Depth of every row (root 0); used to pick per-depth draft inputs."""
    dep = np.zeros(len(parents), dtype=np.int64)
    for i in range(1, len(parents)):
        dep[i] = dep[parents[i]] + 1
    return dep


def prefix_tokens(vocab: int, prefix: int, seed: int = 2) -> np.ndarray:
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 0])))
    return g.integers(0, vocab, size=prefix, dtype=np.int64).astype(np.int32)


def softmax_rows(logits: np.ndarray) -> np.ndarray:
    """Normalised draft distributions from draft logits (input generation)."""
    z = logits.astype(np.float64)
    z = z - z.max(axis=-1, keepdims=True)
    e = np.exp(z)
    return (e / e.sum(axis=-1, keepdims=True)).astype(np.float32)


def draft_q(n_rows: int, vocab: int, q_temp: float, seed: int = 2,
            shared_root_children: np.ndarray | None = None) -> np.ndarray:
    """Draft distributions q[i] (row 0 unused) = softmax(N(0,1)/q_temp).

    If ``shared_root_children`` lists the root's children, they share one q
    row: they are i.i.d. draws from the draft's distribution at the branch
    point.
    """
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 1])))
    lg = g.standard_normal((n_rows, vocab), dtype=np.float32) / np.float32(q_temp)
    q = softmax_rows(lg)
    q[0] = 0.0
    if shared_root_children is not None and len(shared_root_children) > 1:
        q[shared_root_children[1:]] = q[shared_root_children[0]]
    return q


def draw_tokens(q: np.ndarray, seed: int = 2) -> np.ndarray:
    """Draft token of every row i >= 1 drawn from q[i]; row 0 gets -1."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 2])))
    toks = np.full(q.shape[0], -1, dtype=np.int32)
    for i in range(1, q.shape[0]):
        p = q[i].astype(np.float64)
        p /= p.sum()
        toks[i] = g.choice(q.shape[1], p=p)
    return toks


def uniforms(n: int, seed: int = 1) -> np.ndarray:
    return np.random.Generator(np.random.Philox(seed)).random(n, dtype=np.float32)


def random_logits(n_rows: int, vocab: int, scale: float = 2.0, seed: int = 5) -> np.ndarray:
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 3])))
    return (g.standard_normal((n_rows, vocab), dtype=np.float32) * np.float32(scale))


def synthetic_kv(shape: Shape, layer: int, kv_len: int, capacity: int, which: int,
                 seed: int = 3, as_bits: bool = False) -> np.ndarray:
    """Seeded N(0,1) prefix K (which=0) or V (which=1) of one layer,
    [n_kv_heads][capacity][head_dim]; rows >= kv_len are zero."""
    n = shape.n_kv_heads * kv_len * shape.head_dim
    buf = np.empty(n, dtype=np.float32)
    _normal_chunks([seed, layer, which], n, buf)
    buf = buf.reshape(shape.n_kv_heads, kv_len, shape.head_dim)
    if shape.dtype == "bf16":
        out = np.zeros((shape.n_kv_heads, capacity, shape.head_dim), dtype=np.uint16)
        out[:, :kv_len] = bf16_bits(buf)
        return out if as_bits else bits_to_f32(out)
    out = np.zeros((shape.n_kv_heads, capacity, shape.head_dim), dtype=np.float32)
    out[:, :kv_len] = buf
    return out


def step_inputs(w: Workload, seed_tokens: int = 2, seed_u: int = 1) -> dict:
    """Tokens, parents, q and uniforms of one verify step of workload w.

    The root row carries the last prefix token; its KV is written by the
    step itself (the prefix KV holds the first P-1 tokens).
    """
    s = w.shape
    parents = branch_parents(w.branches, w.depth)
    n = len(parents)
    ptoks = prefix_tokens(s.vocab, w.prefix, seed_tokens)
    root_children = np.nonzero(parents == 0)[0]
    q = draft_q(n, s.vocab, w.q_temp, seed_tokens, root_children)
    toks = draw_tokens(q, seed_tokens)
    toks[0] = ptoks[-1]
    return {
        "prefix_tokens": ptoks,
        "parents": parents,
        "tokens": toks,
        "q": q,
        "u": uniforms(n, seed_u),
    }
