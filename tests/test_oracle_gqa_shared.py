"""Pins of the oracle's GQA-shared mode (one selection per KV group): the group's query score
stream is the elementwise max of its heads' streams (combined with the KV head's stream by
the max of Eq. topk); every query head of the group attends over the group's gathered K~, V~;
dK~, dV~ of the group sum over its query heads."""
import numpy as np
import pytest

import oracle
import brute


def _inputs(B, N, Hq, Hkv, D, seed, same_heads=False):
    rng = np.random.default_rng(seed)
    rb = np.vectorize(oracle.round_bf16)
    q = rb(rng.standard_normal((B, N, Hq, D)))
    if same_heads:
        G = Hq // Hkv
        for g in range(Hkv):
            for t in range(1, G):
                q[:, :, g * G + t] = q[:, :, g * G]
    k = rb(rng.standard_normal((B, N, Hkv, D)))
    # a few strong keys so that the KV stream matters in the ranking, and strong rows of each
    # query head at its own positions so that the heads disagree
    k[:, rng.choice(N, 3, replace=False)] *= 4
    if not same_heads:
        for hq in range(Hq):
            q[:, rng.choice(N, 4, replace=False), hq] *= 4
    v = rb(rng.standard_normal((B, N, Hkv, D)))
    return q, k, v


def test_shared_is_per_head_when_each_group_has_one_head():
    q, k, v = _inputs(1, 256, 2, 2, 16, 1)
    a = oracle.layer_forward(q, k, v, 4, 3, 8)
    b = oracle.layer_forward(q, k, v, 4, 3, 8, flags=oracle.GQA_SHARED)
    for key in ("idx", "slot", "qs", "ks", "vs", "os", "lse", "o"):
        np.testing.assert_array_equal(b[key], a[key], err_msg=key)
    dout = np.random.default_rng(2).standard_normal(q.shape)
    ga, gb = oracle.layer_backward(a, dout), oracle.layer_backward(b, dout)
    for key in ("dq", "dk", "dv"):
        np.testing.assert_array_equal(gb[key], ga[key], err_msg=key)


def test_shared_is_per_head_when_the_group_heads_are_equal():
    """Equal query heads select the same entries on their own, so sharing changes nothing; the
    group's dK, dV (gradient of the shared rows summed, then the adjoint) equal the per-head
    sums of adjoints."""
    q, k, v = _inputs(1, 256, 4, 2, 16, 3, same_heads=True)
    a = oracle.layer_forward(q, k, v, 4, 3, 6)
    b = oracle.layer_forward(q, k, v, 4, 3, 6, flags=oracle.GQA_SHARED)
    G = 2
    for hq in range(4):
        np.testing.assert_array_equal(b["idx"][0, hq // G], a["idx"][0, hq])
        np.testing.assert_array_equal(b["ks"][0, hq // G], a["ks"][0, hq])
    for key in ("qs", "os", "lse", "o"):
        np.testing.assert_array_equal(b[key], a[key], err_msg=key)
    dout = np.random.default_rng(4).standard_normal(q.shape)
    ga, gb = oracle.layer_backward(a, dout), oracle.layer_backward(b, dout)
    np.testing.assert_array_equal(gb["dq"], ga["dq"])
    for key in ("dk", "dv"):
        np.testing.assert_allclose(gb[key], ga[key], rtol=1e-12, atol=1e-12, err_msg=key)


@pytest.mark.parametrize("seed", [5, 6, 7])
def test_group_selection_is_the_concatenated_stream_walk(seed):
    N, Hq, Hkv, D, p, L, kk = 256, 3, 1, 16, 4, 4, 5
    q, k, v = _inputs(1, N, Hq, Hkv, D, seed)
    f = oracle.layer_forward(q, k, v, p, L, kk, flags=oracle.GQA_SHARED)
    heads = [brute.level_scores_fsum(q[0, :, hq], p, L) for hq in range(Hq)]
    kv = brute.level_scores_fsum(k[0, :, 0], p, L)
    emitted = brute.select_group_stream(heads, kv, p, L, kk)
    order = brute.causal_sorted(emitted, N, p, L)
    offs, _ = brute.level_offsets(N, p, L)
    np.testing.assert_array_equal(f["idx"][0, 0], [offs[l] + i for l, i in order])
    # the group stream must matter: some head alone would pick differently
    per_head = oracle.layer_forward(q, k, v, p, L, kk)
    assert any(not np.array_equal(per_head["idx"][0, hq], f["idx"][0, 0]) for hq in range(Hq))


def test_shared_adjoint_identity_pins_the_group_sum():
    """With the selection fixed and unrounded pooled rows, O is linear in V, so
    sum over heads <dO, O> = <dV, V>. Dropping any head from the group sum breaks it."""
    q, k, v = _inputs(1, 128, 3, 1, 8, 8)
    f = oracle.layer_forward(q, k, v, 4, 3, 4, dtype=oracle.F64, flags=oracle.GQA_SHARED)
    dout = np.random.default_rng(9).standard_normal(q.shape)
    g = oracle.layer_backward(f, dout)
    lhs = float((dout * f["o"]).sum())
    rhs = float((g["dv"] * v).sum())
    assert abs(lhs - rhs) <= 1e-9 * max(1.0, abs(lhs))


def test_shared_dk_matches_finite_differences():
    q, k, v = _inputs(1, 64, 2, 1, 8, 10)
    p, L, kk = 2, 3, 3
    f = oracle.layer_forward(q, k, v, p, L, kk, dtype=oracle.F64, flags=oracle.GQA_SHARED)
    dout = np.random.default_rng(11).standard_normal(q.shape)
    g = oracle.layer_backward(f, dout)
    rng = np.random.default_rng(12)
    eps = 1e-6
    for _ in range(6):
        j, c = int(rng.integers(64)), int(rng.integers(8))
        kp, km = k.copy(), k.copy()
        kp[0, j, 0, c] += eps
        km[0, j, 0, c] -= eps
        fp = oracle.layer_forward(q, kp, v, p, L, kk, dtype=oracle.F64, flags=oracle.GQA_SHARED)
        fm = oracle.layer_forward(q, km, v, p, L, kk, dtype=oracle.F64, flags=oracle.GQA_SHARED)
        if not (np.array_equal(fp["idx"], f["idx"]) and np.array_equal(fm["idx"], f["idx"])):
            continue  # the perturbation moved the selection: not a smooth point
        fd = float((dout * (fp["o"] - fm["o"])).sum()) / (2 * eps)
        assert abs(fd - g["dk"][0, j, 0, c]) <= 1e-6 * max(1.0, abs(fd)), (j, c, fd, g["dk"][0, j, 0, c])
