"""Independent brute-force formulations used to pin the oracle (tiny inputs only).

Nothing here calls the oracle; each function is a different formulation of a step of the
method (arXiv 2605.06554), written so that a mistake in the oracle's version would show.
"""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np


def level_offsets(N, p, L):
    offs, o = [], 0
    for l in range(L):
        offs.append(o)
        o += N // p ** l
    return offs, o


def pool_exact(x, p, l):
    """Eq. pool with exact rational arithmetic: list of level-l rows (Fractions)."""
    w = p ** l
    N, D = len(x), len(x[0])
    return [[sum(Fraction(float(x[i * w + t][c])) for t in range(w)) / w for c in range(D)]
            for i in range(N // w)]


def round_bf16_exact(x: Fraction) -> float:
    """Nearest bf16 value to an exact rational, ties to even (8 significant bits)."""
    if x == 0:
        return 0.0
    ax = abs(x)
    m, e = math.frexp(float(ax))           # float(ax) ~ ax; fix the binade exactly below
    while Fraction(2) ** (e - 1) > ax:
        e -= 1
    while Fraction(2) ** e <= ax:
        e += 1
    ulp = Fraction(2) ** (e - 8)            # ax in [2^(e-1), 2^e): 8 significant bits
    r = round(ax / ulp) * ulp               # round() on a Fraction is half-to-even
    return float(r if x > 0 else -r)


def norms_fsum(x):
    """Eq. score-base with an exactly rounded sum (math.fsum) and sqrt, rounded to fp32."""
    return np.array([np.float32(math.sqrt(math.fsum(float(v) * float(v) for v in row))) for row in x],
                    np.float32)


def maxpool_levels(s0, p, L):
    """Eq. score-pool by reshaping: level l = max over windows of p^l level-0 scores."""
    s0 = np.asarray(s0, np.float32)
    return [s0.reshape(-1, p ** l).max(axis=1) for l in range(L)]


def select_stream(sqk_levels, skq_levels, p, L, k, replace_parents=False):
    """Per-level descent where each level's parents are found by walking the CONCATENATED
    QK and KQ streams (Eq. topk) in (score desc, index asc) order and keeping the first k
    distinct entries. Returns the emitted level-local index sets, one sorted list per level."""
    cand = list(range(len(sqk_levels[L - 1])))
    emitted = [None] * L
    for l in range(L - 1, -1, -1):
        if l == 0:
            emitted[0] = sorted(cand)
            break
        stream = [(float(sqk_levels[l][i]), i) for i in cand] + [(float(skq_levels[l][i]), i) for i in cand]
        stream.sort(key=lambda t: (-t[0], t[1]))
        parents, seen = [], set()
        for _, i in stream:
            if len(parents) >= k:
                break
            if i not in seen:
                seen.add(i)
                parents.append(i)
        emitted[l] = sorted(set(cand) - set(parents)) if replace_parents else sorted(cand)
        cand = sorted(p * i + r for i in parents for r in range(p))
    return emitted


def causal_sorted(emitted, N, p, L):
    """Causal order of Sec. 3.5: (window end asc, coarser level first). Returns [(l, i)]."""
    ent = [(l, i) for l in range(L) for i in emitted[l]]
    ent.sort(key=lambda e: ((e[1] + 1) * p ** e[0] - 1, -e[0]))
    return ent


def causal_sdpa(q, k, v, scale):
    """Plain causal softmax attention over rows, fp64 (Eq. sdpa)."""
    S = len(q)
    a = (q @ k.T) * scale
    a = np.where(np.tril(np.ones((S, S), bool)), a, -np.inf)
    a = a - a.max(axis=1, keepdims=True)
    w = np.exp(a)
    w /= w.sum(axis=1, keepdims=True)
    return w @ v


def all_pyramid_attention(q, k, v, p, L, scale):
    """Cumulative selection with a budget covering every entry emits the whole pyramid. This
    computes that layer with no sort and no index bookkeeping: a double loop over all pyramid
    entries with the visibility predicate end(t) < end(m), or equal ends and level(t) >= level(m),
    then the shifted range sums of Eq. fanout/scatter written as explicit loops.
    q, k, v: [N, D] fp64 (pooled entries are NOT rounded). Returns O [N, D]."""
    N, D = q.shape
    ent = []  # (level, i, end, pooled q, k, v)
    for l in range(L):
        w = p ** l
        for i in range(N // w):
            sl = slice(i * w, (i + 1) * w)
            ent.append((l, i, (i + 1) * w - 1, q[sl].mean(0), k[sl].mean(0), v[sl].mean(0)))
    O = np.zeros((N, D))
    for (lm, im, em, qm, _, _) in ent:
        logits, vals = [], []
        for (lt, it, et, _, kt, vt) in ent:
            if et < em or (et == em and lt >= lm):
                logits.append(scale * float(qm @ kt))
                vals.append(vt)
        logits = np.array(logits)
        wts = np.exp(logits - logits.max())
        om = (wts[:, None] * np.array(vals)).sum(0) / wts.sum()
        w = p ** lm
        for j in range(em, em + w):
            if j < N:
                O[j] += om
    return O


def select_stratified(sqk_levels, skq_levels, p, L, k, chunk):
    """Stratified per-level descent: a level that ranks (k < #candidates) cuts its candidates,
    in index order, into chunks of `chunk`; chunk [s, e) keeps the first
    floor(k e / n) - floor(k s / n) distinct entries of the concatenated QK and KQ streams of
    its own candidates, walked in (score desc, index asc) order. Returns the emitted sets."""
    cand = list(range(len(sqk_levels[L - 1])))
    emitted = [None] * L
    for l in range(L - 1, -1, -1):
        emitted[l] = sorted(cand)
        if l == 0:
            break
        n = len(cand)
        parents = []
        if k >= n:
            parents = list(cand)
        else:
            for s0 in range(0, n, chunk):
                part = cand[s0:s0 + chunk]
                quota = (k * (s0 + len(part))) // n - (k * s0) // n
                stream = [(float(sqk_levels[l][i]), i) for i in part] + [(float(skq_levels[l][i]), i) for i in part]
                stream.sort(key=lambda t: (-t[0], t[1]))
                seen = []
                for _, i in stream:
                    if len(seen) >= quota:
                        break
                    if i not in seen:
                        seen.append(i)
                parents += seen
        cand = sorted(p * i + r for i in parents for r in range(p))
    return emitted


def select_group_stream(sqk_levels_heads, skq_levels, p, L, k):
    """Per-level descent for a selection shared by a KV group: each level's parents are the
    first k DISTINCT entries of the concatenation of every query head's QK stream and the KV
    head's KQ stream, walked in (score desc, index asc) order. Returns the emitted sets."""
    cand = list(range(len(skq_levels[L - 1])))
    emitted = [None] * L
    for l in range(L - 1, -1, -1):
        emitted[l] = sorted(cand)
        if l == 0:
            break
        stream = [(float(sq[l][i]), i) for sq in sqk_levels_heads for i in cand]
        stream += [(float(skq_levels[l][i]), i) for i in cand]
        stream.sort(key=lambda t: (-t[0], t[1]))
        parents, seen = [], set()
        for _, i in stream:
            if len(parents) >= k:
                break
            if i not in seen:
                seen.add(i)
                parents.append(i)
        cand = sorted(p * i + r for i in parents for r in range(p))
    return emitted


def level_scores_fsum(x, p, L):
    """Eqs. score-base / score-pool without the oracle: exact sum of squares (math.fsum), fp64
    sqrt, rounded to fp32, then max over each window. Returns one array per level."""
    s0 = np.array([np.float32(math.sqrt(math.fsum(float(t) * float(t) for t in row))) for row in x],
                  np.float32)
    out = [s0]
    for l in range(1, L):
        w = p ** l
        out.append(s0.reshape(-1, w).max(axis=1))
    return out
