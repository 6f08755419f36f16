"""Pins of the oracle's selection (Eq. topk, Fig. 2 panel 3) and causal ordering (Sec. 3.5)."""
import json
import os

import numpy as np
import pytest

import oracle
import brute
import workloads

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _fan_in(h, idx):
    fan = np.zeros(h.N, int)
    offs = [h.level_offset(l) for l in range(h.L)] + [h.ptot]
    for t in idx:
        l = max(j for j in range(h.L) if offs[j] <= t)
        i = t - offs[l]
        w = h.p ** l
        for j in range((i + 1) * w - 1, min(h.N, (i + 2) * w - 1)):
            fan[j] += 1
    return fan


def test_fig2_selection_panel():
    g = json.load(open(os.path.join(GOLD, "fig2_selection.json")))
    h = oracle.Head(g["N"], 4, g["p"], g["L"], g["k"], oracle.F32)
    s = np.zeros(h.ptot, np.float32)
    s[h.level_offset(2): h.level_offset(2) + 4] = g["level2_scores"]
    for i, v in zip(g["level1_candidates"], g["level1_scores"]):
        s[h.level_offset(1) + i] = v
    idx, slot = oracle.select(h, s, np.zeros_like(s))
    assert len(idx) == g["S"] == h.N // h.p ** (h.L - 1) + (h.L - 1) * h.p * h.k
    # emitted sets per level, straight from the figure
    for l in range(h.L):
        lo, hi = h.level_offset(l), h.level_offset(l) + h.level_rows(l)
        got = sorted(int(t) - lo for t in idx if lo <= t < hi)
        assert got == g["emitted"][str(l)]
    assert idx.tolist() == g["idx"]
    assert _fan_in(h, idx).tolist() == g["fan_in"]
    assert all(slot[t] == m for m, t in enumerate(idx))
    assert (slot >= 0).sum() == len(idx)


def _random_levels(rng, N, p, L, ties=False):
    """Random per-level score streams (not max-pool consistent: selection is tested alone)."""
    h = oracle.Head(N, 4, p, L, 1, oracle.F32)
    if ties:
        s_qk = rng.integers(0, 4, h.ptot).astype(np.float32)
        s_kq = rng.integers(0, 4, h.ptot).astype(np.float32)
    else:
        s_qk = rng.random(h.ptot).astype(np.float32)
        s_kq = rng.random(h.ptot).astype(np.float32)
    lv_qk = [s_qk[h.level_offset(l): h.level_offset(l) + h.level_rows(l)] for l in range(L)]
    lv_kq = [s_kq[h.level_offset(l): h.level_offset(l) + h.level_rows(l)] for l in range(L)]
    return s_qk, s_kq, lv_qk, lv_kq


@pytest.mark.parametrize("N,p,L,k,ties,rep", [
    (64, 2, 4, 3, False, False), (64, 2, 4, 3, True, False), (81, 3, 3, 4, True, False),
    (256, 4, 4, 5, False, False), (256, 4, 4, 5, True, True), (128, 2, 5, 100, True, False),
    (128, 2, 5, 0, False, False), (96, 2, 6, 2, True, True),
])
def test_select_matches_concatenated_stream_bruteforce(N, p, L, k, ties, rep, rng):
    for trial in range(5):
        s_qk, s_kq, lq, lk = _random_levels(rng, N, p, L, ties)
        h = oracle.Head(N, 4, p, L, k, oracle.F32, oracle.REPLACE_PARENTS if rep else 0)
        idx, slot = oracle.select(h, s_qk, s_kq)
        emitted = brute.select_stream(lq, lk, p, L, k, replace_parents=rep)
        order = brute.causal_sorted(emitted, N, p, L)
        assert idx.tolist() == [h.level_offset(l) + i for (l, i) in order]
        assert len(set(idx.tolist())) == len(idx)


def test_tie_break_lower_index_wins():
    # all-equal scores: the lowest-index candidates become parents at every level
    N, p, L, k = 64, 2, 4, 3
    h = oracle.Head(N, 4, p, L, k, oracle.F32)
    s = np.ones(h.ptot, np.float32)
    idx, _ = oracle.select(h, s, s)
    lv = {l: sorted(int(t) - h.level_offset(l) for t in idx
                    if h.level_offset(l) <= t < h.level_offset(l) + h.level_rows(l)) for l in range(L)}
    assert lv[3] == list(range(8))
    assert lv[2] == [0, 1, 2, 3, 4, 5]          # children of parents {0, 1, 2}
    assert lv[1] == [0, 1, 2, 3, 4, 5]          # children of parents {0, 1, 2}
    assert lv[0] == [0, 1, 2, 3, 4, 5]


def test_duplicate_rows_lower_index_wins():
    # two identical level-2 scores competing for the last parent slot
    N, p, L, k = 16, 2, 3, 1
    h = oracle.Head(N, 4, p, L, k, oracle.F32)
    s = np.zeros(h.ptot, np.float32)
    s[h.level_offset(2) + 1] = 5.0
    s[h.level_offset(2) + 3] = 5.0
    idx, _ = oracle.select(h, s, np.zeros_like(s))
    lvl1 = sorted(int(t) - h.level_offset(1) for t in idx if h.level_offset(1) <= t < h.level_offset(2))
    assert lvl1 == [2, 3]


def _S_formula(N, p, L, k):
    """Eq. S-size generalised to budgets larger than the candidate count."""
    cand, S = N // p ** (L - 1), 0
    for _ in range(L - 1):
        S += cand
        cand = p * min(k, cand)
    return S + cand


@pytest.mark.parametrize("cfg", ["c1", "c2", "c3", "c4", "c5"])
def test_S_table(cfg):
    c = workloads.CONFIGS[cfg]
    expect = {"c1": 832, "c2": 13568, "c3": 37888, "c4": 54272, "c5": 119808}[cfg]
    assert _S_formula(c.N, c.p, c.L, c.k) == expect
    if c.N // c.p ** (c.L - 1) >= c.k:
        assert expect == c.N // c.p ** (c.L - 1) + (c.L - 1) * c.p * c.k


def test_worked_example_subsequence_length(rng):
    # Sec. 3.5: N = 10^6, L = 4, p = 4, k = 4096 gives S of about 6.5e4
    N, p, L, k = 10 ** 6, 4, 4, 4096
    h = oracle.Head(N, 4, p, L, k, oracle.F32)
    s = rng.random(h.ptot).astype(np.float32)
    idx, _ = oracle.select(h, s, s)
    assert len(idx) == N // 64 + 3 * 4 * 4096 == 64777
    assert abs(len(idx) - 6.5e4) / 6.5e4 < 0.01


def test_invariants_on_random_scores(rng):
    N, p, L, k = 4096, 4, 4, 100
    h = oracle.Head(N, 4, p, L, k, oracle.F32)
    s_qk, s_kq, _, _ = _random_levels(rng, N, p, L)
    idx, slot = oracle.select(h, s_qk, s_kq)
    fan = _fan_in(h, idx)
    P = p ** (L - 1)
    assert fan.max() <= L                  # Sec. 3.6: fan-in bounded by L
    assert (fan[P - 1:] >= 1).all()        # coarsest level kept whole
    # coarsest level kept whole, and every base token lies in the window of an emitted entry
    cover = np.zeros(N, int)
    for t in idx:
        l = max(j for j in range(L) if h.level_offset(j) <= t)
        i = t - h.level_offset(l)
        cover[i * p ** l:(i + 1) * p ** l] += 1
    assert (cover >= 1).all()
    ends = []
    for t in idx:
        l = max(j for j in range(L) if h.level_offset(j) <= t)
        i = t - h.level_offset(l)
        ends.append((i + 1) * p ** l - 1)
    assert all(a <= b for a, b in zip(ends, ends[1:]))   # causal (topological) order


def test_spikes_are_selected():
    # closed form: with planted keys scaled x8, their KQ scores dominate every window that holds
    # them, and there are fewer spikes than parents at each level, so each spike is emitted at
    # level 0 in every head
    c = workloads.scaled(workloads.CONFIGS["c2"], N=4096, Hq=2, Hkv=2, k=256)
    inp = workloads.make_inputs(c)
    pos = inp["spikes"].numpy()
    assert 0 < len(pos) <= c.k
    h = oracle.Head(c.N, c.D, c.p, c.L, c.k, oracle.BF16)
    for hq in range(c.Hq):
        q = inp["q"][0, :, hq, :].double().numpy()
        k = inp["k"][0, :, hq, :].double().numpy()
        idx, slot = oracle.select(h, oracle.scores(h, q), oracle.scores(h, k))
        assert (slot[pos] >= 0).all()


# ---------------------------------------------------------------- stratified selection (App. D.2)

@pytest.mark.parametrize("N,p,L,k,ties", [
    (8192, 2, 3, 1500, False), (8192, 2, 3, 1500, True), (65536, 4, 2, 3000, False), (6561, 3, 3, 900, True),
])
def test_stratified_matches_bruteforce(N, p, L, k, ties, rng):
    s_qk, s_kq, lq, lk = _random_levels(rng, N, p, L, ties)
    h = oracle.Head(N, 4, p, L, k, oracle.F32, oracle.STRATIFIED)
    idx, slot = oracle.select(h, s_qk, s_kq)
    emitted = brute.select_stratified(lq, lk, p, L, k, oracle.STRAT_CHUNK)
    order = brute.causal_sorted(emitted, N, p, L)
    assert idx.tolist() == [h.level_offset(l) + i for (l, i) in order]
    # the shapes of the exact mode are kept
    h_exact = oracle.Head(N, 4, p, L, k, oracle.F32)
    assert len(idx) == len(oracle.select(h_exact, s_qk, s_kq)[0])


def test_stratified_single_chunk_is_exact(rng):
    # every level ranks at most 2048 candidates: one chunk, the exact top-k
    N, p, L, k = 4096, 4, 4, 100
    s_qk, s_kq, _, _ = _random_levels(rng, N, p, L, True)
    a = oracle.select(oracle.Head(N, 4, p, L, k, oracle.F32, oracle.STRATIFIED), s_qk, s_kq)[0]
    b = oracle.select(oracle.Head(N, 4, p, L, k, oracle.F32), s_qk, s_kq)[0]
    assert a.tolist() == b.tolist()


def test_stratified_every_chunk_contributes():
    # all high scores in the first chunk: the exact top-k takes all of them, the stratified
    # selection takes each chunk's share (8 chunks of 2048 candidates, 375 parents each)
    N, p, L, k = 65536, 4, 2, 3000
    h = oracle.Head(N, 4, p, L, k, oracle.F32, oracle.STRATIFIED)
    s = np.zeros(h.ptot, np.float32)
    s[h.level_offset(1): h.level_offset(1) + 2048] = 1.0 + np.arange(2048, dtype=np.float32)
    idx, _ = oracle.select(h, s, s)
    parents = sorted({int(t) // p for t in idx if t < h.level_offset(1)})
    per_chunk = np.bincount(np.array(parents) // oracle.STRAT_CHUNK, minlength=8)
    assert per_chunk.tolist() == [375] * 8
    exact = oracle.select(oracle.Head(N, 4, p, L, k, oracle.F32), s, s)[0]
    par_exact = sorted({int(t) // p for t in exact if t < h.level_offset(1)})
    assert np.bincount(np.array(par_exact) // oracle.STRAT_CHUNK, minlength=8)[0] == 2048
