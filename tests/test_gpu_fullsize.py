"""Parity at the workloads' full sizes, through the fused entry points the benchmark times.

The oracle cannot run a whole layer at N = 262,144 in a test (its SDPA alone is about 2 fp64
TFLOP per head), so per config these tests check:
  * every head: the fp32 scores, idx, slot and the gathered rows Q~, K~, V~, bit for bit (the
    oracle computes them in full);
  * c4 (the benchmark workload): every row of O~, lse, O and dQ of the four query heads of KV
    group 0, and every row of that KV head's dK and dV, against the oracle's full layer for the
    group (a query head's outputs depend only on that head and its KV head; dK and dV of a KV
    head sum its query heads);
  * c3 and c5: O~, lse, O and dQ at sampled positions spread over the sequence and dK, dV at
    the last base positions, each computed by the oracle one row at a time; at c5 also dK, dV
    at the first base positions, whose gathered keys are seen by every query row.
A sampled base position is compared only once the oracle has evaluated every gathered row it
depends on. That is verified with the oracle itself: running its scatter (or its gather+pool
adjoint) on an indicator of the rows NOT evaluated must give exactly 0 there.
bf16 tensors that miss the raw 2e-2 bar are held to their bf16 floor (parity.py), emulated on
the same rows.
"""
from __future__ import annotations

import math

import numpy as np
import pytest
import torch

import bf16_floor
import oracle
import workloads
from parity import check_close, check_equal, emulated_floor

pytestmark = pytest.mark.gpu

CHUNK = {"c3": 16, "c4": 8, "c5": 4}   # heads per selection test (keeps each test short)
_STATE: dict = {}


def _host(t):
    return np.ascontiguousarray(t.double().cpu().numpy())


def _layer(name):
    """The fused layer of config `name` on device inputs, run once and kept for the tests of
    that config (the previous config's tensors are released first)."""
    if name in _STATE:
        return _STATE[name]
    import paper_2605_06554_amd as lh

    _STATE.clear()
    torch.cuda.empty_cache()
    cfg = workloads.CONFIGS[name]
    print(f"[fullsize] {name}: N={cfg.N} Hq={cfg.Hq} Hkv={cfg.Hkv} p={cfg.p} L={cfg.L} k={cfg.k}", flush=True)
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
    h = oracle.Head(cfg.N, cfg.D, cfg.p, cfg.L, cfg.k, oracle.BF16)
    _STATE[name] = dict(cfg=cfg, inp=inp, st=st, dq=dq, dk=dk, dv=dv, sqk=sqk, skq=skq, h=h,
                        S=st["idx"].shape[2], heads={})
    return _STATE[name]


def _selection_cases():
    out = []
    for name, n in CHUNK.items():
        cfg = workloads.CONFIGS[name]
        for h0 in range(0, cfg.B * cfg.Hq, n):
            out.append((name, h0, min(cfg.B * cfg.Hq, h0 + n)))
    return out


@pytest.mark.parametrize("name,h0,h1", _selection_cases())
def test_full_size_selection_every_head(name, h0, h1):
    """Scores, idx, slot and the gathered rows of heads [h0, h1) (flattened b * Hq + hq)."""
    L = _layer(name)
    cfg, h, st = L["cfg"], L["h"], L["st"]
    G = cfg.Hq // cfg.Hkv
    pooled = {}
    for flat in range(h0, h1):
        b, hq = divmod(flat, cfg.Hq)
        g = hq // G
        qh = _host(L["inp"]["q"][b, :, hq])
        s_qk = oracle.scores(h, qh)
        check_equal(f"{name} s_qk[{b},{hq}]", L["sqk"][b, hq].cpu().numpy(), s_qk)
        if (b, g) not in pooled:
            kh, vh = _host(L["inp"]["k"][b, :, g]), _host(L["inp"]["v"][b, :, g])
            s_kq = oracle.scores(h, kh)
            check_equal(f"{name} s_kq[{b},{g}]", L["skq"][b, g].cpu().numpy(), s_kq)
            pooled = {(b, g): (s_kq, oracle.pool(h, kh), oracle.pool(h, vh))}
            del kh, vh
        s_kq, kpyr, vpyr = pooled[(b, g)]
        idx, slot = oracle.select(h, s_qk, s_kq)
        assert len(idx) == L["S"]
        check_equal(f"{name} idx[{b},{hq}]", st["idx"][b, hq].cpu().numpy(), idx)
        check_equal(f"{name} slot[{b},{hq}]", st["slot"][b, hq].cpu().numpy(), slot)
        check_equal(f"{name} qs[{b},{hq}]", _host(st["qs"][b, hq]), oracle.gather(h, oracle.pool(h, qh), idx))
        check_equal(f"{name} ks[{b},{hq}]", _host(st["ks"][b, hq]), oracle.gather(h, kpyr, idx))
        check_equal(f"{name} vs[{b},{hq}]", _host(st["vs"][b, hq]), oracle.gather(h, vpyr, idx))
    print(f"[fullsize] {name} heads {h0}..{h1 - 1}: selection and gathered rows bit-exact", flush=True)


# ------------------------------------------------------------------ c4: one KV group, every row

C4_GROUP = 0


def _c4_head(hq):
    """The oracle's full layer for query head hq of KV group C4_GROUP (every row), and its bf16
    floor emulation; kept for the dK / dV test."""
    L = _layer("c4")
    if hq in L["heads"]:
        return L["heads"][hq]
    cfg, h = L["cfg"], L["h"]
    G = cfg.Hq // cfg.Hkv
    assert hq // G == C4_GROUP
    sc = 1.0 / math.sqrt(cfg.D)
    qh = _host(L["inp"]["q"][0, :, hq])
    kh, vh = _host(L["inp"]["k"][0, :, C4_GROUP]), _host(L["inp"]["v"][0, :, C4_GROUP])
    f = oracle.head_forward(h, sc, qh, kh, vh)
    del qh, kh, vh
    dout = _host(L["inp"]["dout"][0, :, hq])
    idx = f["idx"]
    dos = oracle.scatter_bwd(h, idx, dout)
    dqs, dks, dvs = oracle.sdpa_bwd(f["qs"], f["ks"], f["vs"], f["os"], f["lse"], dos, sc)
    r = dict(idx=idx, os=f["os"], lse=f["lse"], o=f["o"], dq=oracle.gather_pool_bwd(h, idx, dqs),
             dk=oracle.gather_pool_bwd(h, idx, dks), dv=oracle.gather_pool_bwd(h, idx, dvs))
    # bf16 floor on the same rows
    e_os, e_lse = bf16_floor.sdpa_fwd(f["qs"], f["ks"], f["vs"], sc)
    e_dos = bf16_floor.round_bf16(dos)
    e_dqs, e_dks, e_dvs = bf16_floor.sdpa_bwd(f["qs"], f["ks"], f["vs"], e_os, e_lse, e_dos, sc)
    r["e_os"] = e_os
    r["e_o"] = bf16_floor.round_bf16(oracle.scatter(h, idx, e_os))
    r["e_dq"] = bf16_floor.round_bf16(oracle.gather_pool_bwd(h, idx, e_dqs))
    r["e_dk"] = oracle.gather_pool_bwd(h, idx, bf16_floor.round_bf16(e_dks))
    r["e_dv"] = oracle.gather_pool_bwd(h, idx, bf16_floor.round_bf16(e_dvs))
    L["heads"][hq] = r
    return r


@pytest.mark.timeout(900)
@pytest.mark.parametrize("t", range(4))
def test_c4_group_every_row(t):
    """O~, lse, O and dQ of query head t of KV group 0 at c4, every row."""
    L = _layer("c4")
    hq = C4_GROUP * (L["cfg"].Hq // L["cfg"].Hkv) + t
    r = _c4_head(hq)
    st = L["st"]
    check_close(f"c4 os[0,{hq}]", _host(st["os"][0, hq]), r["os"], "bf16", emulated_floor(r["e_os"], r["os"]))
    check_close(f"c4 lse[0,{hq}]", st["lse"][0, hq].double().cpu().numpy(), r["lse"], "fp32")
    check_close(f"c4 o[0,{hq}]", _host(st["o"][0, :, hq]), r["o"], "bf16", emulated_floor(r["e_o"], r["o"]))
    check_close(f"c4 dq[0,{hq}]", _host(L["dq"][0, :, hq]), r["dq"], "bf16", emulated_floor(r["e_dq"], r["dq"]))
    print(f"[fullsize] c4 head {hq}: every row checked", flush=True)


@pytest.mark.timeout(900)
def test_c4_group_dk_dv_every_row():
    """dK and dV of KV head 0 at c4 (the sums over its four query heads), every base row."""
    L = _layer("c4")
    G = L["cfg"].Hq // L["cfg"].Hkv
    rs = [_c4_head(C4_GROUP * G + t) for t in range(G)]
    for nm in ("dk", "dv"):
        ref = sum(r[nm] for r in rs)
        emu = bf16_floor.round_bf16(sum(r["e_" + nm] for r in rs))
        check_close(f"c4 {nm}[0,{C4_GROUP}]", _host(L[nm][0, :, C4_GROUP]), ref, "bf16", emulated_floor(emu, ref))


# ------------------------------------------------------------------ c3, c5: sampled positions

# (config, heads (b, hq) sampled for O/dQ, KV group (b, g) whose dK/dV are checked, number of
#  sampled base positions, tail rows)
SAMPLED = {
    "c3": ([(0, 0), (1, 31)], (1, 31), 16, 384),
    "c5": ([(0, 0), (0, 15)], (0, 15), 16, 512),
}


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


def _head_inputs(L, b, hq):
    cfg, h = L["cfg"], L["h"]
    g = hq // (cfg.Hq // cfg.Hkv)
    qh, kh, vh = (_host(L["inp"][x][b, :, hh]) for x, hh in (("q", hq), ("k", g), ("v", g)))
    idx = L["st"]["idx"][b, hq].cpu().numpy()   # equal to the oracle's (selection test)
    qs = oracle.gather(h, oracle.pool(h, qh), idx)
    ks = oracle.gather(h, oracle.pool(h, kh), idx)
    vs = oracle.gather(h, oracle.pool(h, vh), idx)
    dos = oracle.scatter_bwd(h, idx, _host(L["inp"]["dout"][b, :, hq]))
    return idx, qs, ks, vs, dos


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", list(SAMPLED))
def test_full_size_sampled_parity(name):
    heads, (gb, gg), n_sample, tail = SAMPLED[name]
    L = _layer(name)
    cfg, h, st, S = L["cfg"], L["h"], L["st"], L["S"]
    sc = 1.0 / math.sqrt(cfg.D)
    rng = np.random.default_rng(7)
    P = cfg.p ** (cfg.L - 1)
    j_sample = np.unique(np.concatenate([
        rng.choice(cfg.N, n_sample, replace=False),
        [0, P - 2, P - 1, cfg.N // 2, cfg.N - 1]]))
    jt_ = torch.as_tensor(j_sample, device="cuda")
    tail_rows = np.arange(S - tail, S)
    for b, hq in heads:
        idx, qs, ks, vs, dos = _head_inputs(L, b, hq)
        # rows the sampled outputs depend on: those whose scatter range [e, e + p^l - 1] or
        # pooling window [e - p^l + 1, e] holds a sampled j (checked below with the oracle)
        e_of, w_of = _window_ends(h, idx)
        need = set(tail_rows.tolist())
        for j in j_sample:
            need.update(np.nonzero((e_of <= j) & (j <= e_of + w_of - 1))[0].tolist())
            need.update(np.nonzero((e_of - w_of + 1 <= j) & (j <= e_of))[0].tolist())
        rows = np.array(sorted(need), np.int64)
        assert not _uncovered(h, idx, rows, S, False)[j_sample].any(), "O sample depends on an unevaluated row"
        assert not _uncovered(h, idx, rows, S, True)[j_sample].any(), "dQ sample depends on an unevaluated row"
        os_ref, lse_ref = oracle.sdpa_fwd(qs, ks, vs, sc, row_list=rows)
        dqs_ref = oracle.sdpa_bwd_dq_rows(qs, ks, vs, os_ref, lse_ref, dos, sc, rows)
        e_os, e_lse = bf16_floor.sdpa_fwd(qs, ks, vs, sc, rows=rows)
        e_dos = bf16_floor.round_bf16(dos)
        e_dqs, _, _ = bf16_floor.sdpa_bwd(qs, ks, vs, e_os, e_lse, e_dos, sc, qrows=rows, krange=(S, S))
        check_close(f"{name} os[{b},{hq}]", _host(st["os"][b, hq])[rows], os_ref[rows], "bf16",
                    emulated_floor(e_os[rows], os_ref[rows]))
        check_close(f"{name} lse[{b},{hq}]", st["lse"][b, hq].double().cpu().numpy()[rows], lse_ref[rows], "fp32")
        o_ref = oracle.scatter(h, idx, os_ref)[j_sample]
        e_o = bf16_floor.round_bf16(oracle.scatter(h, idx, e_os)[j_sample])
        dq_ref = oracle.gather_pool_bwd(h, idx, dqs_ref)[j_sample]
        e_dq = bf16_floor.round_bf16(oracle.gather_pool_bwd(h, idx, e_dqs)[j_sample])
        check_close(f"{name} o[{b},{hq}]", _host(st["o"][b, :, hq][jt_]), o_ref, "bf16", emulated_floor(e_o, o_ref))
        check_close(f"{name} dq[{b},{hq}]", _host(L["dq"][b, :, hq][jt_]), dq_ref, "bf16", emulated_floor(e_dq, dq_ref))
        print(f"[fullsize] {name} head ({b},{hq}): {len(rows)} rows evaluated", flush=True)
    # dK, dV of the checked KV group at the last base positions (G = 1 at c3 and c5)
    assert cfg.Hq == cfg.Hkv
    idx, qs, ks, vs, dos = _head_inputs(L, gb, gg)
    os_ref, lse_ref = oracle.sdpa_fwd(qs, ks, vs, sc, rows=(S - tail, S))
    _, dks, dvs = oracle.sdpa_bwd(qs, ks, vs, os_ref, lse_ref, dos, sc, qrows=(S, S), krows=(S - tail, S))
    e_os, e_lse = bf16_floor.sdpa_fwd(qs, ks, vs, sc, rows=tail_rows)
    _, e_dks, e_dvs = bf16_floor.sdpa_bwd(qs, ks, vs, e_os, e_lse, bf16_floor.round_bf16(dos), sc, qrows=[],
                                          krange=(S - tail, S))
    unc = _uncovered(h, idx, tail_rows, S, True)
    jt = np.arange(cfg.N - 256, cfg.N)
    jt = jt[unc[jt] == 0]
    assert len(jt) >= 64, f"only {len(jt)} tail positions are fully evaluated"
    _check_dkdv(name, L, gb, gg, idx, jt, dks, dvs, e_dks, e_dvs)


def _check_dkdv(name, L, b, g, idx, jt, dks, dvs, e_dks, e_dvs):
    h = L["h"]
    jt_ = torch.as_tensor(jt, device="cuda")
    for nm, ref_s, emu_s in (("dk", dks, e_dks), ("dv", dvs, e_dvs)):
        ref = oracle.gather_pool_bwd(h, idx, ref_s)[jt]
        emu = bf16_floor.round_bf16(oracle.gather_pool_bwd(h, idx, bf16_floor.round_bf16(emu_s))[jt])
        check_close(f"{name} {nm}[{b},{g}] ({len(jt)} positions)", _host(L[nm][b, :, g][jt_]), ref, "bf16",
                    emulated_floor(emu, ref))


@pytest.mark.timeout(900)
def test_c5_first_keys_dk_dv():
    """dK, dV at the first base positions of KV head 15 at c5. Their gathered keys are attended
    by every later query row, so the oracle runs the full forward of the head (all 119,808
    rows) and the key adjoint of the first gathered rows."""
    L = _layer("c5")
    cfg, h, S = L["cfg"], L["h"], L["S"]
    b, g = 0, 15
    sc = 1.0 / math.sqrt(cfg.D)
    idx, qs, ks, vs, dos = _head_inputs(L, b, g)
    T = 512
    os_ref, lse_ref = oracle.sdpa_fwd(qs, ks, vs, sc)
    _, dks, dvs = oracle.sdpa_bwd(qs, ks, vs, os_ref, lse_ref, dos, sc, qrows=(S, S), krows=(0, T))
    # floor: the storage roundings of O~ and dO~ and the roundings of P and dS on these rows
    _, e_dks, e_dvs = bf16_floor.sdpa_bwd(qs, ks, vs, bf16_floor.round_bf16(os_ref), lse_ref,
                                          bf16_floor.round_bf16(dos), sc, qrows=[], krange=(0, T))
    unc = _uncovered(h, idx, np.arange(T), S, True)
    jt = np.nonzero(unc == 0)[0]
    jt = jt[jt < cfg.N // 2]
    assert len(jt) >= 64, f"only {len(jt)} leading positions depend on the first {T} gathered rows alone"
    _check_dkdv("c5 first", L, b, g, idx, jt, dks, dvs, e_dks, e_dvs)
    print(f"[fullsize] c5 first keys: {len(jt)} base positions checked", flush=True)
