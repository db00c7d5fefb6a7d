"""The verify step's softmax statistics are summed per block of 16 logits
relative to the block's own largest scaled logit and rescaled to the row's
(the LM head's epilogue folds its logits that way).  This CPU check states
that arithmetic in numpy -- float32 scaled logits and exponentials, float64
sums, exp(m_b - zmax) from the exact float64 difference through the float
exponential and a first-order correction -- and holds it to the row
statistics' definition (oracle.sampling.row_stats): zmax and argmax exact,
total within 1e-7 relative, NaN where the definition gives NaN, on rows
with ties, masked (-inf) entries, NaN and +inf entries, all-masked rows and
T = 0."""
import math

import numpy as np
import pytest

from oracle import sampling

f32 = np.float32


def exp_diff(x, y):
    d = float(x) - float(y)
    if d < -104.0:
        return 0.0
    dh = f32(d)
    with np.errstate(over="ignore", invalid="ignore"):
        return float(np.exp(dh)) * (1.0 + (d - float(dh)))


def block(x, c0, V, inv_t, greedy):
    best, arg, bad = -np.inf, None, False
    for j, v in enumerate(x):
        if c0 + j >= V:
            break
        bad |= bool(np.isnan(v) or v == np.inf)
        if v > best:
            best, arg = v, c0 + j
    s = 0.0
    if bad:
        s = math.nan
    elif not greedy and best > -np.inf:
        m = f32(f32(best) * inv_t)
        with np.errstate(invalid="ignore", over="ignore"):
            for j, v in enumerate(x[:V - c0]):
                s += float(np.exp(f32(f32(v) * inv_t) - m))
    return [f32(best), arg, s]


def merge(r, p, inv_t, greedy):
    old = r[0]
    if p[0] > r[0] or (p[0] == r[0] and p[1] is not None and (r[1] is None or p[1] < r[1])):
        r[0], r[1] = p[0], p[1]
    if greedy:
        r[2] += p[2]
        return
    if p[2] == 0.0:
        return
    mo, mp = f32(f32(old) * inv_t), f32(f32(p[0]) * inv_t)
    if mp > mo:
        r[2] = r[2] * exp_diff(mo, mp) + p[2]
    else:
        r[2] += p[2] * exp_diff(mp, mo)


def block_stats(l, T, groups):
    V = len(l)
    greedy = T <= 0
    inv_t = f32(1.0) if greedy else f32(1.0) / f32(T)
    tiles = (V + 15) // 16
    parts = []
    for g in range(groups):
        r = [f32(-np.inf), None, 0.0]
        for t in range(tiles * g // groups, tiles * (g + 1) // groups):
            merge(r, block(l[t * 16:t * 16 + 16], t * 16, V, inv_t, greedy), inv_t, greedy)
        parts.append(r)
    best, arg = -np.inf, None
    for p in parts:
        if p[0] > best or (p[0] == best and p[1] is not None and (arg is None or p[1] < arg)):
            best, arg = p[0], p[1]
    zmax = f32(best) if greedy else f32(f32(best) * inv_t)
    total = 0.0
    for p in parts:
        total += p[2] if greedy or p[2] == 0.0 else p[2] * exp_diff(f32(f32(p[0]) * inv_t), zmax)
    if greedy:
        total = math.nan if math.isnan(total) else 1.0
    elif best == -np.inf:
        total = math.nan
    return zmax, (0 if arg is None else arg), total


CASES = []
for V, T, groups in [(1000, 1.0, 7), (32000, 0.7, 250), (1001, 0.0, 13), (37, 1.3, 3),
                     (2052, 0.9, 17), (4096, 2.0, 64)]:
    for kind in ("plain", "masked", "nan", "all_masked", "ties", "posinf"):
        CASES.append((V, T, groups, kind))


@pytest.mark.parametrize("V,T,groups,kind", CASES)
def test_block_statistics_match_the_definition(V, T, groups, kind):
    rng = np.random.default_rng(V + groups + len(kind))
    l = (rng.standard_normal(V) * 3).astype(f32)
    if kind == "masked":
        l[rng.integers(0, V, V // 3)] = -np.inf
    elif kind == "nan":
        l[V // 2] = np.nan
    elif kind == "all_masked":
        l[:] = -np.inf
    elif kind == "ties":
        l[[3, V // 2, V - 1]] = l.max() + 1.0
    elif kind == "posinf":
        l[V // 3] = np.inf
    rs = sampling.row_stats(l, T)
    zmax, arg, total = block_stats(l, T, groups)
    assert np.float32(zmax) == np.float32(rs.zmax)
    assert arg == rs.argmax
    if math.isnan(rs.total):
        assert math.isnan(total)
    else:
        assert abs(total - rs.total) <= 1e-7 * rs.total
