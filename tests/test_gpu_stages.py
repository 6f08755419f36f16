"""Per-stage parity of the HIP path against the oracle (small shapes, several tiles, ragged
tails). Every call goes through the C ABI."""
import json
import os

import numpy as np
import pytest
import torch

import bf16_floor
import oracle
import workloads
from parity import check_close, check_equal, emulated_floor, rounding_floor, to64

lh = pytest.importorskip("paper_2605_06554_amd")

pytestmark = pytest.mark.gpu
GOLD = os.path.join(os.path.dirname(__file__), "golden")
DEV = "cuda"


def _cfg(name):
    return {**workloads.CONFIGS, **workloads.TEST_CONFIGS}[name]


def _problem(c, **kw):
    d = dict(B=c.B, N=c.N, Hq=c.Hq, Hkv=c.Hkv, D=c.D, p=c.p, L=c.L, k=c.k,
             dtype=lh.LH_BF16 if c.dtype == "bf16" else lh.LH_F32, scale=0.0, flags=c.flags)
    d.update(kw)
    return lh.problem(**d)


def _odt(c):
    return oracle.BF16 if c.dtype == "bf16" else oracle.F32


STAGE_CFGS = ["c1", "t_gqa", "t_f32", "t_p3", "t_k0", "t_l2", "t_l2g", "t_p3g", "t_p5g", "t_l8", "t_g3",
              "t_grp4", "t_grp_tail", "t_grp_f32", "t_grp_wide"]


@pytest.mark.parametrize("name", STAGE_CFGS + ["t_l1"])
def test_pool_and_score(name):
    c = _cfg(name)
    print(f"[stage pool/score] {name}", flush=True)
    inp = workloads.make_inputs(c, with_grad=False)
    pr = _problem(c)
    Ptot = lh.lh_pyramid_rows(pr)
    R = Ptot - c.N
    q, k, v = (inp[x].to(DEV) for x in ("q", "k", "v"))
    dt = q.dtype
    qp = torch.empty(c.B, max(R, 1), c.Hq, c.D, dtype=dt, device=DEV)
    kp = torch.empty(c.B, max(R, 1), c.Hkv, c.D, dtype=dt, device=DEV)
    vp = torch.empty_like(kp)
    sqk = torch.empty(c.B, c.Hq, Ptot, dtype=torch.float32, device=DEV)
    skq = torch.empty(c.B, c.Hkv, Ptot, dtype=torch.float32, device=DEV)
    lh.lh_pyramid_pool(pr, q, k, v, qp, kp, vp)
    lh.lh_score(pr, q, k, sqk, skq)
    # the fused single pass must write exactly the same bytes
    qp2, kp2, vp2, sqk2, skq2 = (torch.empty_like(t) for t in (qp, kp, vp, sqk, skq))
    lh.lh_pool_score(pr, q, k, v, qp2, kp2, vp2, sqk2, skq2)
    torch.cuda.synchronize()
    assert torch.equal(sqk, sqk2) and torch.equal(skq, skq2)
    if R > 0:
        assert torch.equal(qp, qp2) and torch.equal(kp, kp2) and torch.equal(vp, vp2)
    h = oracle.Head(c.N, c.D, c.p, c.L, c.k, _odt(c))
    for b in range(c.B):
        for hh in range(c.Hq):
            x = inp["q"][b, :, hh, :].double().numpy()
            check_equal(f"s_qk[{b},{hh}]", sqk[b, hh], oracle.scores(h, x))
            if R > 0:
                check_equal(f"qpyr[{b},{hh}]", to64(qp[b, :, hh]), oracle.pool(h, x)[c.N:])
        for hh in range(c.Hkv):
            xk = inp["k"][b, :, hh, :].double().numpy()
            xv = inp["v"][b, :, hh, :].double().numpy()
            check_equal(f"s_kq[{b},{hh}]", skq[b, hh], oracle.scores(h, xk))
            if R > 0:
                check_equal(f"kpyr[{b},{hh}]", to64(kp[b, :, hh]), oracle.pool(h, xk)[c.N:])
                check_equal(f"vpyr[{b},{hh}]", to64(vp[b, :, hh]), oracle.pool(h, xv)[c.N:])


def _run_select(pr, sqk, skq):
    S, Ptot = lh.lh_subseq_len(pr), lh.lh_pyramid_rows(pr)
    idx = torch.empty(pr.B, pr.Hq, S, dtype=torch.int32, device=DEV)
    slot = torch.empty(pr.B, pr.Hq, Ptot, dtype=torch.int32, device=DEV)
    ws = lh.workspace(pr, lh.LH_OP_SELECT)
    lh.lh_select_topk(pr, sqk, skq, idx, slot, ws)
    torch.cuda.synchronize()
    return idx.cpu().numpy(), slot.cpu().numpy()


def test_select_fig2_toy():
    g = json.load(open(os.path.join(GOLD, "fig2_selection.json")))
    pr = lh.problem(1, g["N"], 1, 1, 64, g["p"], g["L"], g["k"], lh.LH_F32)
    Ptot = lh.lh_pyramid_rows(pr)
    s = np.zeros(Ptot, np.float32)
    off1, off2 = lh.lh_level_offset(pr, 1), lh.lh_level_offset(pr, 2)
    s[off2: off2 + 4] = g["level2_scores"]
    for i, v in zip(g["level1_candidates"], g["level1_scores"]):
        s[off1 + i] = v
    sq = torch.from_numpy(s).view(1, 1, Ptot).to(DEV)
    sk = torch.zeros_like(sq)
    idx, slot = _run_select(pr, sq, sk)
    assert idx[0, 0].tolist() == g["idx"]
    assert all(slot[0, 0, t] == m for m, t in enumerate(g["idx"]))
    assert (slot >= 0).sum() == g["S"]


@pytest.mark.parametrize("ties", [False, True])
@pytest.mark.parametrize("N,p,L,k,flags", [(4096, 4, 4, 100, 0), (4096, 4, 4, 100, 1), (2048, 2, 6, 37, 0),
                                           (2187, 3, 3, 50, 1), (16384, 4, 5, 4096, 0), (65536, 4, 3, 8192, 0),
                                           # stratified: several chunks of 2048 candidates per level
                                           (65536, 4, 3, 8192, 2), (65536, 4, 2, 3000, 2), (8192, 2, 3, 1500, 3),
                                           (6561, 3, 3, 900, 2),
                                           # levels of 40,000 and 131,072 candidates: keys in the
                                           # workspace instead of LDS
                                           (262144, 4, 3, 10000, 0), (262144, 4, 3, 10000, 2),
                                           (262144, 2, 2, 50000, 1),
                                           # several ranges of 8,192 window ends in the order
                                           # kernel that split coarse windows (p = 3, 5), with
                                           # and without replace mode
                                           (19683, 3, 4, 500, 1), (20000, 5, 3, 300, 0),
                                           (20000, 5, 3, 300, 1), (59049, 3, 3, 3000, 3)])
def test_select_random_scores(N, p, L, k, flags, ties, rng):
    Hq, Hkv = 4, 2
    print(f"[stage select] N={N} p={p} L={L} k={k} flags={flags} ties={ties}", flush=True)
    pr = lh.problem(2, N, Hq, Hkv, 64, p, L, k, lh.LH_F32, 0.0, flags)
    Ptot = lh.lh_pyramid_rows(pr)
    if ties:
        sq = rng.integers(0, 5, (2, Hq, Ptot)).astype(np.float32)
        sk = rng.integers(0, 5, (2, Hkv, Ptot)).astype(np.float32)
    else:
        sq = rng.random((2, Hq, Ptot)).astype(np.float32)
        sk = rng.random((2, Hkv, Ptot)).astype(np.float32)
    idx, slot = _run_select(pr, torch.from_numpy(sq).to(DEV), torch.from_numpy(sk).to(DEV))
    h = oracle.Head(N, 64, p, L, k, oracle.F32, flags)
    for b in range(2):
        for hq in range(Hq):
            ri, rs = oracle.select(h, sq[b, hq], sk[b, hq // 2])
            check_equal(f"idx[{b},{hq}]", idx[b, hq], ri)
            check_equal(f"slot[{b},{hq}]", slot[b, hq], rs)


@pytest.mark.parametrize("kind", ["constant", "low_bits", "wide", "zeros"])
@pytest.mark.parametrize("N,p,L,k,flags", [(16384, 4, 5, 4096, 0), (65536, 4, 3, 8192, 2), (4096, 4, 4, 100, 1),
                                           (262144, 4, 3, 10000, 0)])
def test_select_key_bit_patterns(kind, N, p, L, k, flags, rng):
    # Score patterns that drive the radix select's digit choice to its edges: every key equal
    # (no digit pass at all), keys that differ only in the lowest mantissa bits (one short
    # final digit), keys spanning many binades (a first digit at the sign/exponent byte),
    # and mostly-zero scores with a few positive ones.
    Hq, Hkv = 4, 2
    print(f"[stage select bits] kind={kind} N={N} p={p} L={L} k={k} flags={flags}", flush=True)
    pr = lh.problem(2, N, Hq, Hkv, 64, p, L, k, lh.LH_F32, 0.0, flags)
    Ptot = lh.lh_pyramid_rows(pr)
    shape_q, shape_k = (2, Hq, Ptot), (2, Hkv, Ptot)
    if kind == "constant":
        sq, sk = np.full(shape_q, 3.25, np.float32), np.full(shape_k, 3.25, np.float32)
    elif kind == "low_bits":
        base = np.uint32(np.float32(1.5).view(np.uint32))
        sq = (base + rng.integers(0, 8, shape_q).astype(np.uint32)).view(np.float32)
        sk = (base + rng.integers(0, 8, shape_k).astype(np.uint32)).view(np.float32)
    elif kind == "wide":
        sq = (2.0 ** rng.uniform(-60, 60, shape_q)).astype(np.float32)
        sk = (2.0 ** rng.uniform(-60, 60, shape_k)).astype(np.float32)
    else:
        sq = np.where(rng.random(shape_q) < 0.01, rng.random(shape_q), 0.0).astype(np.float32)
        sk = np.zeros(shape_k, np.float32)
    idx, slot = _run_select(pr, torch.from_numpy(sq).to(DEV), torch.from_numpy(sk).to(DEV))
    h = oracle.Head(N, 64, p, L, k, oracle.F32, flags)
    for b in range(2):
        for hq in range(Hq):
            ri, rs = oracle.select(h, sq[b, hq], sk[b, hq // 2])
            check_equal(f"idx[{b},{hq}]", idx[b, hq], ri)
            check_equal(f"slot[{b},{hq}]", slot[b, hq], rs)


def test_select_large_levels_from_scores():
    """The c5 shape (N = 1,048,576, p = 4, L = 6) with k = 16,384: levels 2 and 1 rank 65,536
    candidates each, beyond the LDS key buffer. Scores from lh_pool_score on device inputs, then
    lh_select_topk; scores, idx and slot against the oracle, bit for bit."""
    c = workloads.scaled(workloads.CONFIGS["c5"], Hq=2, Hkv=2, k=16384, name="c5-k16384")
    print("[stage select] c5 shape with k = 16384", flush=True)
    pr = _problem(c)
    S, Ptot = lh.lh_subseq_len(pr), lh.lh_pyramid_rows(pr)
    assert S == 1024 + 4096 + 16384 + 3 * 65536
    inp = workloads.make_inputs(c, device=DEV, with_grad=False)
    q, k, v = inp["q"], inp["k"], inp["v"]
    R = Ptot - c.N
    qp = torch.empty(c.B, R, c.Hq, c.D, dtype=q.dtype, device=DEV)
    kp, vp = torch.empty(c.B, R, c.Hkv, c.D, dtype=q.dtype, device=DEV), torch.empty(c.B, R, c.Hkv, c.D, dtype=q.dtype, device=DEV)
    sqk = torch.empty(c.B, c.Hq, Ptot, dtype=torch.float32, device=DEV)
    skq = torch.empty(c.B, c.Hkv, Ptot, dtype=torch.float32, device=DEV)
    lh.lh_pool_score(pr, q, k, v, qp, kp, vp, sqk, skq)
    idx, slot = _run_select(pr, sqk, skq)
    h = oracle.Head(c.N, c.D, c.p, c.L, c.k, oracle.BF16)
    for hq in range(c.Hq):
        s_qk = oracle.scores(h, np.ascontiguousarray(q[0, :, hq].double().cpu().numpy()))
        s_kq = oracle.scores(h, np.ascontiguousarray(k[0, :, hq].double().cpu().numpy()))
        check_equal(f"s_qk[{hq}]", sqk[0, hq], s_qk)
        check_equal(f"s_kq[{hq}]", skq[0, hq], s_kq)
        ri, rs = oracle.select(h, s_qk, s_kq)
        check_equal(f"idx[{hq}]", idx[0, hq], ri)
        check_equal(f"slot[{hq}]", slot[0, hq], rs)


def _layer_oracle(c, inp):
    q, k, v = (inp[x].double().numpy() for x in ("q", "k", "v"))
    return oracle.layer_forward(q, k, v, c.p, c.L, c.k, dtype=_odt(c), flags=c.flags)


@pytest.mark.parametrize("name", STAGE_CFGS)
def test_gather_sdpa_scatter_stages(name):
    c = _cfg(name)
    print(f"[stage gather/sdpa/scatter] {name}", flush=True)
    inp = workloads.make_inputs(c)
    f = _layer_oracle(c, inp)
    g = oracle.layer_backward(f, inp["dout"].double().numpy())
    pr = _problem(c)
    S, Ptot = lh.lh_subseq_len(pr), lh.lh_pyramid_rows(pr)
    R = Ptot - c.N
    dt = inp["q"].dtype
    q, k, v, dout = (inp[x].to(DEV) for x in ("q", "k", "v", "dout"))
    qp = torch.empty(c.B, max(R, 1), c.Hq, c.D, dtype=dt, device=DEV)
    kp = torch.empty(c.B, max(R, 1), c.Hkv, c.D, dtype=dt, device=DEV)
    vp = torch.empty_like(kp)
    lh.lh_pyramid_pool(pr, q, k, v, qp, kp, vp)
    idx = torch.from_numpy(f["idx"].astype(np.int32)).to(DEV)
    slot = torch.from_numpy(f["slot"].astype(np.int32)).to(DEV)
    qs, ks, vs, os_ = (torch.empty(c.B, c.Hq, S, c.D, dtype=dt, device=DEV) for _ in range(4))
    lh.lh_gather(pr, q, k, v, qp, kp, vp, idx, qs, ks, vs)
    torch.cuda.synchronize()
    check_equal("qs", to64(qs), f["qs"])
    check_equal("ks", to64(ks), f["ks"])
    check_equal("vs", to64(vs), f["vs"])
    lse = torch.empty(c.B, c.Hq, S, dtype=torch.float32, device=DEV)
    lh.lh_sdpa_fwd(pr, qs, ks, vs, os_, lse)
    torch.cuda.synchronize()
    sc = f["scale"]
    bf = c.dtype == "bf16"
    os_emu = {}
    for b in range(c.B):
        for hq in range(c.Hq):
            fl = None
            if bf:
                os_emu[b, hq], _ = bf16_floor.sdpa_fwd(f["qs"][b, hq], f["ks"][b, hq], f["vs"][b, hq], sc)
                fl = emulated_floor(os_emu[b, hq], f["os"][b, hq])
            check_close(f"os[{b},{hq}]", os_[b, hq], f["os"][b, hq], c.dtype, fl)
            check_close(f"lse[{b},{hq}]", lse[b, hq], f["lse"][b, hq], "fp32")
    # scatter of the oracle's own sub-sequence output (rounded to the dtype) isolates the scatter
    os_ref_h = torch.from_numpy(f["os"]).to(dt)
    os_ref = os_ref_h.to(DEV)
    o = torch.empty_like(q)
    lh.lh_scatter(pr, os_ref, slot, o)
    torch.cuda.synchronize()
    h = f["head"]
    for b in range(c.B):
        for hq in range(c.Hq):
            ref = oracle.scatter(h, f["idx"][b, hq], to64(os_ref[b, hq]))
            check_close(f"o[{b},{hq}]", o[b, :, hq], ref, c.dtype, rounding_floor(ref) if bf else None)
    dos = torch.empty(c.B, c.Hq, S, c.D, dtype=dt, device=DEV)
    lh.lh_scatter_bwd(pr, dout, slot, dos)
    torch.cuda.synchronize()
    for b in range(c.B):
        for hq in range(c.Hq):
            check_close(f"dos[{b},{hq}]", dos[b, hq], g["dos"][b, hq], c.dtype,
                        rounding_floor(g["dos"][b, hq]) if bf else None)
    # SDPA backward on the oracle's inputs: its os rounded to the dtype, its lse, and its dos
    # rounded to the dtype. The floor emulation takes the same rounded os: with planted key
    # spikes, dQ~ depends on the rounding of os through Delta = rowsum(dO~ * O~) amplified by
    # the spiked keys, so the GPU forward's own os (another valid rounding) would make the
    # backward's error a different sample from the emulated one.
    dqs, dks, dvs = (torch.empty(c.B, c.Hq, S, c.D, dtype=dt, device=DEV) for _ in range(3))
    dos_ref = torch.from_numpy(g["dos"]).to(dt).to(DEV)
    lse_ref = torch.from_numpy(np.asarray(f["lse"], np.float32)).to(DEV)
    ws = lh.workspace(pr, lh.LH_OP_SDPA_BWD)
    lh.lh_sdpa_bwd(pr, qs, ks, vs, os_ref, lse_ref, dos_ref, dqs, dks, dvs, ws)
    torch.cuda.synchronize()
    for b in range(c.B):
        for hq in range(c.Hq):
            args = (f["qs"][b, hq], f["ks"][b, hq], f["vs"][b, hq])
            rq, rk, rv = oracle.sdpa_bwd(*args, f["os"][b, hq], f["lse"][b, hq], to64(dos_ref[b, hq]), sc)
            fq = fk = fv = None
            if bf:
                eq, ek, ev = bf16_floor.sdpa_bwd(*args, os_ref_h[b, hq].double().numpy(), f["lse"][b, hq],
                                                 to64(dos_ref[b, hq]), sc)
                fq = emulated_floor(eq, rq)
                fk = emulated_floor(bf16_floor.round_bf16(ek), rk)
                fv = emulated_floor(bf16_floor.round_bf16(ev), rv)
            check_close(f"dqs[{b},{hq}]", dqs[b, hq], rq, c.dtype, fq)
            check_close(f"dks[{b},{hq}]", dks[b, hq], rk, c.dtype, fk)
            check_close(f"dvs[{b},{hq}]", dvs[b, hq], rv, c.dtype, fv)
    # gather + pool backward on the oracle's sub-sequence gradients
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    dqs_r, dks_r, dvs_r = (torch.from_numpy(g[x]).to(dt).to(DEV) for x in ("dqs", "dks", "dvs"))
    lh.lh_gather_bwd(pr, dqs_r, dks_r, dvs_r, slot, dq, dk, dv)
    torch.cuda.synchronize()
    G = c.Hq // c.Hkv
    for b in range(c.B):
        for hq in range(c.Hq):
            ref = oracle.gather_pool_bwd(h, f["idx"][b, hq], to64(dqs_r[b, hq]))
            check_close(f"dq[{b},{hq}]", dq[b, :, hq], ref, c.dtype, rounding_floor(ref) if bf else None)
        for gg in range(c.Hkv):
            rk = np.zeros((c.N, c.D))
            rv = np.zeros((c.N, c.D))
            for hq in range(gg * G, (gg + 1) * G):
                oracle.gather_pool_bwd(h, f["idx"][b, hq], to64(dks_r[b, hq]), rk)
                oracle.gather_pool_bwd(h, f["idx"][b, hq], to64(dvs_r[b, hq]), rv)
            check_close(f"dk[{b},{gg}]", dk[b, :, gg], rk, c.dtype, rounding_floor(rk) if bf else None)
            check_close(f"dv[{b},{gg}]", dv[b, :, gg], rv, c.dtype, rounding_floor(rv) if bf else None)


@pytest.mark.parametrize("S,D,dt", [(1, 128, "bf16"), (31, 64, "bf16"), (300, 128, "bf16"), (1000, 64, "bf16"),
                                    (2113, 128, "bf16"), (257, 64, "fp32"), (700, 128, "fp32")])
def test_sdpa_standalone(S, D, dt, rng):
    print(f"[stage sdpa] S={S} D={D} {dt}", flush=True)
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    B, H = 1, 2
    pr = lh.problem(B, S, H, H, D, 2, 1, 0, tdt)  # L = 1: S rows
    assert lh.lh_subseq_len(pr) == S
    x = [torch.from_numpy(rng.standard_normal((B, H, S, D))).to(tdt) for _ in range(4)]
    qs, ks, vs, dos = (t.to(DEV) for t in x)
    os_ = torch.empty_like(qs)
    lse = torch.empty(B, H, S, dtype=torch.float32, device=DEV)
    lh.lh_sdpa_fwd(pr, qs, ks, vs, os_, lse)
    dqs, dks, dvs = torch.empty_like(qs), torch.empty_like(qs), torch.empty_like(qs)
    ws = lh.workspace(pr, lh.LH_OP_SDPA_BWD)
    lh.lh_sdpa_bwd(pr, qs, ks, vs, os_, lse, dos, dqs, dks, dvs, ws)
    torch.cuda.synchronize()
    sc = 1.0 / np.sqrt(D)
    for hh in range(H):
        a = [t[0, hh].double().numpy() for t in x]
        ro, rl = oracle.sdpa_fwd(a[0], a[1], a[2], sc)
        fo = fq = fk = fv = None
        if dt == "bf16":
            eo, _ = bf16_floor.sdpa_fwd(a[0], a[1], a[2], sc)
            fo = emulated_floor(eo, ro)
        check_close(f"os[{hh}]", os_[0, hh], ro, dt, fo)
        check_close(f"lse[{hh}]", lse[0, hh], rl, "fp32")
        rq, rk, rv = oracle.sdpa_bwd(a[0], a[1], a[2], ro, rl, a[3], sc)
        if dt == "bf16":
            eq, ek, ev = bf16_floor.sdpa_bwd(a[0], a[1], a[2], eo, rl, a[3], sc)
            fq = emulated_floor(eq, rq)
            fk = emulated_floor(bf16_floor.round_bf16(ek), rk)
            fv = emulated_floor(bf16_floor.round_bf16(ev), rv)
        check_close(f"dqs[{hh}]", dqs[0, hh], rq, dt, fq)
        check_close(f"dks[{hh}]", dks[0, hh], rk, dt, fk)
        check_close(f"dvs[{hh}]", dvs[0, hh], rv, dt, fv)
