"""Pins of the oracle's gather / SDPA / scatter chain and its backward.

Special cases that reduce to a library routine (torch SDPA in fp64), the all-pyramid brute
force, the k = 0 closed form, causality, finite differences and adjoint identities."""
import numpy as np
import pytest
import torch

import oracle
import brute


def _torch_causal_sdpa(q, k, v, scale):
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a))[None, None]
    return torch.nn.functional.scaled_dot_product_attention(
        t(q), t(k), t(v), is_causal=True, scale=scale)[0, 0].numpy()


def _rand(rng, *shape):
    return rng.standard_normal(shape)


def test_L1_is_causal_sdpa(rng):
    B, N, Hq, Hkv, D = 2, 50, 4, 2, 16
    q, k, v = _rand(rng, B, N, Hq, D), _rand(rng, B, N, Hkv, D), _rand(rng, B, N, Hkv, D)
    f = oracle.layer_forward(q, k, v, p=4, L=1, kk=0, dtype=oracle.F64)
    sc = 1 / np.sqrt(D)
    for b in range(B):
        for hq in range(Hq):
            ref = _torch_causal_sdpa(q[b, :, hq], k[b, :, hq // 2], v[b, :, hq // 2], sc)
            assert np.allclose(f["o"][b, :, hq], ref, rtol=0, atol=1e-12)
            assert f["idx"][b, hq].tolist() == list(range(N))


@pytest.mark.parametrize("p,L", [(2, 3), (4, 3), (3, 2)])
def test_replace_mode_full_budget_is_causal_sdpa(p, L, rng):
    N, D = p ** (L - 1) * 6, 8
    q, k, v = _rand(rng, 1, N, 1, D), _rand(rng, 1, N, 1, D), _rand(rng, 1, N, 1, D)
    f = oracle.layer_forward(q, k, v, p=p, L=L, kk=N, dtype=oracle.F64, flags=oracle.REPLACE_PARENTS)
    assert f["idx"][0, 0].tolist() == list(range(N))   # only level 0 remains, in order
    ref = _torch_causal_sdpa(q[0, :, 0], k[0, :, 0], v[0, :, 0], 1 / np.sqrt(D))
    assert np.allclose(f["o"][0, :, 0], ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("p,L,N", [(2, 3, 16), (4, 3, 64), (3, 3, 27), (2, 4, 24)])
def test_full_budget_equals_all_pyramid_bruteforce(p, L, N, rng):
    D = 8
    q, k, v = _rand(rng, 1, N, 1, D), _rand(rng, 1, N, 1, D), _rand(rng, 1, N, 1, D)
    f = oracle.layer_forward(q, k, v, p=p, L=L, kk=N, dtype=oracle.F64)
    h = f["head"]
    assert f["idx"].shape[-1] == h.ptot
    ref = brute.all_pyramid_attention(q[0, :, 0], k[0, :, 0], v[0, :, 0], p, L, 1 / np.sqrt(D))
    assert np.allclose(f["o"][0, :, 0], ref, rtol=0, atol=1e-12)


def test_k0_is_coarsest_level_attention(rng):
    # k = 0: only the coarsest level is gathered; O_j = Otilde_i for i = floor((j+1)/P) - 1
    N, p, L, D = 96, 2, 4, 8
    P = p ** (L - 1)
    q, k, v = _rand(rng, 1, N, 1, D), _rand(rng, 1, N, 1, D), _rand(rng, 1, N, 1, D)
    f = oracle.layer_forward(q, k, v, p=p, L=L, kk=0, dtype=oracle.F64)
    pool = lambda x: x[0, :, 0].reshape(N // P, P, D).mean(1)
    ot = brute.causal_sdpa(pool(q), pool(k), pool(v), 1 / np.sqrt(D))
    ref = np.zeros((N, D))
    for j in range(P - 1, N):
        ref[j] = ot[(j + 1) // P - 1]
    assert np.allclose(f["o"][0, :, 0], ref, rtol=0, atol=1e-12)


def _forward_fixed(h, sc, q, k, v, idx):
    qs = oracle.gather(h, oracle.pool(h, q), idx)
    ks = oracle.gather(h, oracle.pool(h, k), idx)
    vs = oracle.gather(h, oracle.pool(h, v), idx)
    os_, lse = oracle.sdpa_fwd(qs, ks, vs, sc)
    return oracle.scatter(h, idx, os_), (qs, ks, vs, os_, lse)


def test_causality_with_fixed_selection(rng):
    N, p, L, D, kk = 256, 4, 4, 16, 6
    q, k, v = _rand(rng, 1, N, 1, D), _rand(rng, 1, N, 1, D), _rand(rng, 1, N, 1, D)
    f = oracle.layer_forward(q, k, v, p=p, L=L, kk=kk, dtype=oracle.BF16)
    t = 150
    # flip signs of Q and K rows after t and redraw V after t: norms (hence the selection)
    # are unchanged, and outputs up to t must be bit-identical
    q2, k2, v2 = q.copy(), k.copy(), v.copy()
    q2[:, t + 1:] *= -1
    k2[:, t + 1:] *= -1
    v2[:, t + 1:] = _rand(rng, 1, N - t - 1, 1, D)
    g = oracle.layer_forward(q2, k2, v2, p=p, L=L, kk=kk, dtype=oracle.BF16)
    assert np.array_equal(f["idx"], g["idx"])
    assert np.array_equal(f["o"][:, : t + 1], g["o"][:, : t + 1])
    assert not np.array_equal(f["o"][:, t + 1:], g["o"][:, t + 1:])


def test_finite_differences_with_fixed_selection(rng):
    # dL/dq, dk, dv of L = <dout, O> by central differences with the selection held fixed,
    # pooled entries stored unrounded (fp64), GQA with two query heads on one KV head
    N, p, L, D, kk, Hq = 32, 2, 3, 6, 3, 2
    q, k, v = _rand(rng, 1, N, Hq, D), _rand(rng, 1, N, 1, D), _rand(rng, 1, N, 1, D)
    dout = _rand(rng, 1, N, Hq, D)
    f = oracle.layer_forward(q, k, v, p=p, L=L, kk=kk, dtype=oracle.F64)
    gr = oracle.layer_backward(f, dout)
    h, sc = f["head"], f["scale"]

    def loss(q_, k_, v_):
        tot = 0.0
        for hq in range(Hq):
            o, _ = _forward_fixed(h, sc, np.ascontiguousarray(q_[0, :, hq]), np.ascontiguousarray(k_[0, :, 0]),
                                  np.ascontiguousarray(v_[0, :, 0]), f["idx"][0, hq])
            tot += float((o * dout[0, :, hq]).sum())
        return tot

    eps = 1e-5
    for name, arr, grad in (("q", q, gr["dq"]), ("k", k, gr["dk"]), ("v", v, gr["dv"])):
        for _ in range(12):
            j, hh, c = rng.integers(N), rng.integers(arr.shape[2]), rng.integers(D)
            a, b = arr.copy(), arr.copy()
            a[0, j, hh, c] += eps
            b[0, j, hh, c] -= eps
            args_a = {"q": (a, k, v), "k": (q, a, v), "v": (q, k, a)}[name]
            args_b = {"q": (b, k, v), "k": (q, b, v), "v": (q, k, b)}[name]
            fd = (loss(*args_a) - loss(*args_b)) / (2 * eps)
            assert abs(fd - grad[0, j, hh, c]) <= 1e-6 * max(1.0, abs(fd)), (name, j, hh, c)


def test_sdpa_bwd_matches_autograd(rng):
    S, D = 40, 8
    qs, ks, vs, dos = (_rand(rng, S, D) for _ in range(4))
    sc = 0.3
    os_, lse = oracle.sdpa_fwd(qs, ks, vs, sc)
    dq, dk, dv = oracle.sdpa_bwd(qs, ks, vs, os_, lse, dos, sc)
    t = [torch.from_numpy(a.copy())[None, None].requires_grad_(True) for a in (qs, ks, vs)]
    o = torch.nn.functional.scaled_dot_product_attention(*t, is_causal=True, scale=sc)
    o.backward(torch.from_numpy(dos)[None, None])
    for mine, ref in ((dq, t[0].grad), (dk, t[1].grad), (dv, t[2].grad)):
        assert np.allclose(mine, ref[0, 0].numpy(), rtol=0, atol=1e-12)
    ref_lse = torch.logsumexp(torch.from_numpy(
        np.where(np.tril(np.ones((S, S), bool)), sc * qs @ ks.T, -np.inf)), dim=1).numpy()
    assert np.allclose(lse, ref_lse, rtol=0, atol=1e-12)
    # row subsets agree with the full computation
    o2, l2 = oracle.sdpa_fwd(qs, ks, vs, sc, rows=(30, 40))
    assert np.array_equal(o2[30:], os_[30:]) and np.array_equal(l2[30:], lse[30:])
    _, dk2, dv2 = oracle.sdpa_bwd(qs, ks, vs, os_, lse, dos, sc, qrows=(0, 0), krows=(35, 40))
    assert np.array_equal(dk2[35:], dk[35:]) and np.array_equal(dv2[35:], dv[35:])


def test_adjoint_identities(rng):
    N, p, L, D, kk = 128, 4, 4, 8, 5
    h = oracle.Head(N, D, p, L, kk, oracle.F64)
    s = rng.random(h.ptot).astype(np.float32)
    idx, slot = oracle.select(h, s, s)
    S = len(idx)
    X, Y = _rand(rng, S, D), _rand(rng, N, D)
    # <scatter(X), Y> = <X, scatter_bwd(Y)>
    assert np.isclose((oracle.scatter(h, idx, X) * Y).sum(), (X * oracle.scatter_bwd(h, idx, Y)).sum(),
                      rtol=1e-12, atol=0)
    # <gather(pool(Z)), W> = <Z, gather_pool_bwd(W)>
    Z, W = _rand(rng, N, D), _rand(rng, S, D)
    lhs = (oracle.gather(h, oracle.pool(h, Z), idx) * W).sum()
    rhs = (Z * oracle.gather_pool_bwd(h, idx, W)).sum()
    assert np.isclose(lhs, rhs, rtol=1e-12, atol=0)


def test_output_linear_in_v(rng):
    # O is linear in V for fixed Q, K and selection, hence <dout, O> = <dV, V>
    N, p, L, D, kk, Hq = 64, 2, 4, 8, 4, 2
    q, k, v = _rand(rng, 1, N, Hq, D), _rand(rng, 1, N, 1, D), _rand(rng, 1, N, 1, D)
    dout = _rand(rng, 1, N, Hq, D)
    f = oracle.layer_forward(q, k, v, p=p, L=L, kk=kk, dtype=oracle.F64)
    g = oracle.layer_backward(f, dout)
    assert np.isclose((dout * f["o"]).sum(), (g["dv"] * v).sum(), rtol=1e-10, atol=0)


def test_row_list_sdpa_matches_full_rows(rng):
    """The sampled-row SDPA entry points give the same rows as the full computation."""
    S, D = 300, 16
    qs, ks, vs, dos = (rng.standard_normal((S, D)) for _ in range(4))
    sc = 0.25
    os_full, lse_full = oracle.sdpa_fwd(qs, ks, vs, sc)
    dq_full, _, _ = oracle.sdpa_bwd(qs, ks, vs, os_full, lse_full, dos, sc)
    rows = np.array([0, 1, 57, 150, 298, 299])
    os_r, lse_r = oracle.sdpa_fwd(qs, ks, vs, sc, row_list=rows)
    assert np.array_equal(os_r[rows], os_full[rows]) and np.array_equal(lse_r[rows], lse_full[rows])
    other = np.setdiff1d(np.arange(S), rows)
    assert not os_r[other].any() and not lse_r[other].any()
    dq_r = oracle.sdpa_bwd_dq_rows(qs, ks, vs, os_r, lse_r, dos, sc, rows)
    assert np.array_equal(dq_r[rows], dq_full[rows]) and not dq_r[other].any()
