"""Pins of the oracle's pooling (Eq. pool) and scoring (Eqs. score-base, score-pool)."""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
import brute

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def test_bf16_rounding_matches_library_cast(rng):
    # fp64 values exactly representable in fp32: rounding to bf16 must equal torch's
    # fp32 -> bf16 conversion (round to nearest, ties to even).
    x32 = (rng.standard_normal(20000) * np.exp(rng.uniform(-20, 20, 20000))).astype(np.float32)
    ties = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8), 2 ** -130, 3.0 * 2 ** -9 + 1], np.float32)
    x32 = np.concatenate([x32, ties])
    ref = torch.from_numpy(x32).to(torch.bfloat16).to(torch.float64).numpy()
    got = np.array([oracle.round_bf16(float(v)) for v in x32])
    assert np.array_equal(got, ref)


def test_pool_exact_on_dyadic_inputs(rng):
    # Dyadic inputs make every fp64 sum exact, so the oracle must equal exact rational means.
    N, D, p, L = 48, 3, 2, 4
    x = rng.integers(-64, 64, (N, D)).astype(np.float64) / 8.0
    h = oracle.Head(N, D, p, L, 1, oracle.F64)
    pyr = oracle.pool(h, x)
    for l in range(L):
        off = h.level_offset(l)
        exact = brute.pool_exact(x, p, l)
        for i, row in enumerate(exact):
            assert [float(v) for v in row] == pyr[off + i].tolist()


@pytest.mark.parametrize("p,L", [(2, 4), (3, 3), (4, 3)])
def test_pool_closed_forms(p, L):
    # constant rows pool to the same constant; a ramp x_j = j*u pools to (i p^l + (p^l-1)/2) u
    N, D = p ** (L - 1) * 5, 4
    u = np.array([1.0, -2.0, 0.5, 3.0])
    h = oracle.Head(N, D, p, L, 1, oracle.F64)
    const = np.full((N, D), 1.75)
    assert np.all(oracle.pool(h, const) == 1.75)
    ramp = np.arange(N, dtype=np.float64)[:, None] * u[None, :]
    pyr = oracle.pool(h, ramp)
    for l in range(L):
        w = p ** l
        for i in range(N // w):
            expect = (i * w + (w - 1) / 2.0) * u
            assert np.allclose(pyr[h.level_offset(l) + i], expect, rtol=0, atol=1e-12)


def test_pool_bf16_storage_rounds_exact_mean(rng):
    N, D, p, L = 64, 8, 4, 3
    x = torch.randn(N, D).to(torch.bfloat16).double().numpy()
    h = oracle.Head(N, D, p, L, 1, oracle.BF16)
    pyr = oracle.pool(h, x)
    for l in range(1, L):
        exact = brute.pool_exact(x, p, l)
        for i, row in enumerate(exact):
            ref = [brute.round_bf16_exact(v) for v in row]
            assert pyr[h.level_offset(l) + i].tolist() == ref


def test_norm_of_pythagorean_rows():
    h = oracle.Head(4, 6, 2, 1, 0, oracle.F32)
    x = np.zeros((4, 6))
    x[0, :2] = (3, 4)
    x[1, 2:4] = (5, 12)
    x[2, :] = 1.0
    x[3, 5] = -7.0
    s = oracle.scores(h, x)
    assert s.tolist() == [5.0, 13.0, np.float32(math.sqrt(6.0)), 7.0]


def test_fig2_norm_score_panel():
    g = json.load(open(os.path.join(GOLD, "fig2_norm_score.json")))
    p, L = g["p"], g["L"]
    s0 = g["level0"]
    N = len(s0)
    x = np.zeros((N, 4))
    x[:, 0] = s0  # rows s * e1 have norm exactly s
    h = oracle.Head(N, 4, p, L, 1, oracle.F32)
    s = oracle.scores(h, x)
    assert s[: N].tolist() == s0
    assert s[h.level_offset(1): h.level_offset(2)].tolist() == g["level1"]
    assert s[h.level_offset(2): h.ptot].tolist() == g["level2"]


@pytest.mark.parametrize("dt", ["fp32", "bf16"])
def test_scores_match_fsum_and_maxpool(dt, rng):
    N, D, p, L = 256, 64, 4, 4
    t = torch.from_numpy(rng.standard_normal((N, D)) * 3)
    t = t.float() if dt == "fp32" else t.to(torch.bfloat16)
    x = t.double().numpy()
    h = oracle.Head(N, D, p, L, 1, oracle.F32)
    s = oracle.scores(h, x)
    s0 = brute.norms_fsum(x)
    if dt == "bf16":
        # squares of bf16 values are short, so the fp64 sum is exact in any order
        assert np.array_equal(s[:N], s0)
    else:
        assert np.max(np.abs(s[:N].astype(np.float64) - s0) / s0) <= 2 ** -23
    lv = brute.maxpool_levels(s[:N], p, L)
    for l in range(1, L):
        assert np.array_equal(s[h.level_offset(l): h.level_offset(l) + N // p ** l], lv[l])


def test_pyramid_size_bound():
    # Sec. 3.3: sum_l N/p^l <= N p/(p-1)
    for (N, p, L) in [(4096, 4, 5), (2 ** 20, 4, 6), (2187, 3, 7), (1024, 2, 11)]:
        h = oracle.Head(N, 8, p, L, 1)
        assert h.ptot == sum(N // p ** l for l in range(L))
        assert h.ptot <= N * p / (p - 1)


def test_check_rejects_indivisible():
    assert oracle.Head(1000, 8, 4, 4, 1).check() == -2   # 64 does not divide 1000
    assert oracle.Head(1024, 8, 4, 4, 1).check() == 0
    assert oracle.Head(1024, 8, 1, 2, 1).check() == -3
    assert oracle.Head(1024, 8, 4, 0, 1).check() == -3
