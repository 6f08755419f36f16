"""Parity at the workloads' full sizes, through the fused entry points the benchmark times.

The oracle cannot run a whole layer at N = 262,144 (the SDPA alone is about 2 fp64 TFLOP per
head), so these tests check, per config:
  * scores, idx and slot of every checked head bit for bit (the oracle computes them in full);
  * the gathered rows Q~, K~, V~ of those heads bit for bit;
  * O~, lse, O and dQ at sampled positions spread over the sequence, and dK, dV at the last
    base positions, each computed by the oracle one row at a time.
A sampled base position is compared only once the oracle has evaluated every gathered row it
depends on. That is verified with the oracle itself: running its scatter (or its gather+pool
adjoint) on an indicator of the rows NOT evaluated must give exactly 0 there.
"""
from __future__ import annotations

import math

import numpy as np
import pytest
import torch

import oracle
import workloads
from parity import check_close, check_equal

pytestmark = pytest.mark.gpu

# (config, heads (b, hq) checked in full for scores/selection/gather and sampled for O/dQ,
#  KV group (b, g) whose dK/dV are checked, number of sampled base positions, tail rows)
CASES = {
    # the benchmark workload: GQA 32/8, spikes, S = 54,272
    "c4": (workloads.CONFIGS["c4"], [(0, 0), (0, 31)], (0, 0), 24, 384),
    # B = 2 and near-tied scores in a rank-64 subspace, S = 37,888
    "c3": (workloads.CONFIGS["c3"], [(0, 0), (1, 31)], (1, 31), 16, 384),
    # the largest shape: N = 1,048,576, L = 6, 32,768 candidates per level (the selection limit)
    "c5": (workloads.CONFIGS["c5"], [(0, 0), (0, 15)], (0, 15), 16, 512),
}


def _host(t):
    return np.ascontiguousarray(t.double().cpu().numpy())


def _run_layer(cfg):
    import paper_2605_06554_amd as lh

    inp = workloads.make_inputs(cfg, device="cuda")
    q, k, v, dout = inp["q"], inp["k"], inp["v"], inp["dout"]
    pr, st = lh.attention_forward(q, k, v, cfg.p, cfg.L, cfg.k)
    dq, dk, dv = lh.attention_backward(pr, st, dout)
    Ptot = lh.lh_pyramid_rows(pr)
    # scores through their own entry point: the fused pass runs the same kernel on the same input
    sqk = torch.empty(cfg.B, cfg.Hq, Ptot, dtype=torch.float32, device="cuda")
    skq = torch.empty(cfg.B, cfg.Hkv, Ptot, dtype=torch.float32, device="cuda")
    lh.lh_score(pr, q, k, sqk, skq)
    torch.cuda.synchronize()
    return inp, st, dict(dq=dq, dk=dk, dv=dv, sqk=sqk, skq=skq)


def _window_ends(h, idx):
    """Window end e = (i + 1) p^l - 1 and width p^l of every gathered entry (flattened id
    off_l + i)."""
    offs = np.array([h.level_offset(l) for l in range(h.L)], np.int64)
    ids = idx.astype(np.int64)
    lvl = np.searchsorted(offs, ids, side="right") - 1
    w = np.asarray(h.p, np.int64) ** lvl
    return (ids - offs[lvl] + 1) * w - 1, w


def _uncovered(h, idx, known_rows, S, adjoint):
    """Per base position: nonzero iff the scatter (adjoint=False) or the gather+pool adjoint
    (adjoint=True) of the oracle reads a gathered row outside known_rows."""
    ind = np.ones((S, 1), np.float64)
    ind[known_rows] = 0.0
    ind = np.ascontiguousarray(np.repeat(ind, h.D, axis=1))
    if adjoint:
        out = oracle.gather_pool_bwd(h, idx, ind)
    else:
        out = oracle.scatter(h, idx, ind)
    return np.abs(out).max(axis=1)


@pytest.mark.parametrize("name", list(CASES))
def test_full_size_sampled_parity(name):
    cfg, heads, (gb, gg), n_sample, tail = CASES[name]
    print(f"[fullsize] {name}: N={cfg.N} Hq={cfg.Hq} Hkv={cfg.Hkv} p={cfg.p} L={cfg.L} k={cfg.k}", flush=True)
    inp, st, out = _run_layer(cfg)
    G = cfg.Hq // cfg.Hkv
    sc = 1.0 / math.sqrt(cfg.D)
    h = oracle.Head(cfg.N, cfg.D, cfg.p, cfg.L, cfg.k, oracle.BF16)
    S = st["idx"].shape[2]
    rng = np.random.default_rng(7)
    P = cfg.p ** (cfg.L - 1)
    j_sample = np.unique(np.concatenate([
        rng.choice(cfg.N, n_sample, replace=False),
        [0, P - 2, P - 1, cfg.N // 2, cfg.N - 1]]))
    group_heads = [(gb, gb_h) for gb_h in range(gg * G, gg * G + G)]
    todo = list(dict.fromkeys(heads + group_heads))
    dk_ref = np.zeros((cfg.N, cfg.D))
    dv_ref = np.zeros((cfg.N, cfg.D))
    dkv_unc = np.zeros(cfg.N)
    tail_rows = np.arange(S - tail, S)
    for b, hq in todo:
        g = hq // G
        qh, kh, vh = _host(inp["q"][b, :, hq]), _host(inp["k"][b, :, g]), _host(inp["v"][b, :, g])
        # scores, selection and the gathered rows: in full, bit for bit
        s_qk, s_kq = oracle.scores(h, qh), oracle.scores(h, kh)
        check_equal(f"{name} s_qk[{b},{hq}]", out["sqk"][b, hq].cpu().numpy(), s_qk)
        check_equal(f"{name} s_kq[{b},{g}]", out["skq"][b, g].cpu().numpy(), s_kq)
        idx, slot = oracle.select(h, s_qk, s_kq)
        assert len(idx) == S
        check_equal(f"{name} idx[{b},{hq}]", st["idx"][b, hq].cpu().numpy(), idx)
        check_equal(f"{name} slot[{b},{hq}]", st["slot"][b, hq].cpu().numpy(), slot)
        qs = oracle.gather(h, oracle.pool(h, qh), idx)
        ks = oracle.gather(h, oracle.pool(h, kh), idx)
        vs = oracle.gather(h, oracle.pool(h, vh), idx)
        for nm, ref in (("qs", qs), ("ks", ks), ("vs", vs)):
            check_equal(f"{name} {nm}[{b},{hq}]", _host(st[nm][b, hq]), ref)
        del qh
        # rows the sampled outputs depend on: those whose scatter range [e, e + p^l - 1] or
        # pooling window [e - p^l + 1, e] holds a sampled j (checked below with the oracle)
        e_of, w_of = _window_ends(h, idx)
        need = set(tail_rows.tolist())
        for j in j_sample:
            need.update(np.nonzero((e_of <= j) & (j <= e_of + w_of - 1))[0].tolist())
            need.update(np.nonzero((e_of - w_of + 1 <= j) & (j <= e_of))[0].tolist())
        rows = np.array(sorted(need), np.int64)
        os_ref, lse_ref = oracle.sdpa_fwd(qs, ks, vs, sc, row_list=rows)
        dout_h = _host(inp["dout"][b, :, hq])
        dos_ref = oracle.scatter_bwd(h, idx, dout_h)
        del dout_h
        dqs_ref = oracle.sdpa_bwd_dq_rows(qs, ks, vs, os_ref, lse_ref, dos_ref, sc, rows)
        # gathered-level outputs of the forward at the evaluated rows
        check_close(f"{name} os[{b},{hq}]", _host(st["os"][b, hq])[rows], os_ref[rows], "bf16")
        check_close(f"{name} lse[{b},{hq}]", st["lse"][b, hq].double().cpu().numpy()[rows], lse_ref[rows], "fp32")
        # base-level O and dQ at the sampled positions
        o_ref = oracle.scatter(h, idx, os_ref)
        dq_ref = oracle.gather_pool_bwd(h, idx, dqs_ref)
        assert not _uncovered(h, idx, rows, S, False)[j_sample].any(), "O sample depends on an unevaluated row"
        assert not _uncovered(h, idx, rows, S, True)[j_sample].any(), "dQ sample depends on an unevaluated row"
        jt_ = torch.as_tensor(j_sample, device="cuda")
        check_close(f"{name} o[{b},{hq}]", _host(st["o"][b, :, hq][jt_]), o_ref[j_sample], "bf16")
        check_close(f"{name} dq[{b},{hq}]", _host(out["dq"][b, :, hq][jt_]), dq_ref[j_sample], "bf16")
        # dK, dV of the checked KV group: tail rows of every query head of the group
        if (b, hq) in group_heads:
            _, dks, dvs = oracle.sdpa_bwd(qs, ks, vs, os_ref, lse_ref, dos_ref, sc, qrows=(S, S),
                                          krows=(S - tail, S))
            oracle.gather_pool_bwd(h, idx, dks, dk_ref)
            oracle.gather_pool_bwd(h, idx, dvs, dv_ref)
            dkv_unc += _uncovered(h, idx, tail_rows, S, True)
        print(f"[fullsize] {name} head ({b},{hq}) ok: {len(rows)} rows evaluated", flush=True)
    # base positions at the end whose dK/dV depend only on the evaluated tail rows of every head
    jt = np.arange(cfg.N - 256, cfg.N)
    jt = jt[dkv_unc[jt] == 0]
    assert len(jt) >= 64, f"only {len(jt)} tail positions are fully evaluated"
    jt_ = torch.as_tensor(jt, device="cuda")
    check_close(f"{name} dk[{gb},{gg}]", _host(out["dk"][gb, :, gg][jt_]), dk_ref[jt], "bf16")
    check_close(f"{name} dv[{gb},{gg}]", _host(out["dv"][gb, :, gg][jt_]), dv_ref[jt], "bf16")
