"""The gather fused into the SDPA loads (lh_*_indexed): outputs must be bitwise identical to the
materialised path (lh_gather + lh_sdpa_fwd / lh_sdpa_bwd), which the other GPU tests compare with
the oracle; one case is also compared with the oracle directly."""
import numpy as np
import pytest
import torch

import oracle
import workloads
from parity import check_close_heads, check_equal, check_layer

lh = pytest.importorskip("paper_2605_06554_amd")

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _cfg(name):
    return {**workloads.CONFIGS, **workloads.TEST_CONFIGS}[name]


def _same(name, a, b):
    assert a.shape == b.shape, (name, a.shape, b.shape)
    ai = a.contiguous().view(torch.int16 if a.element_size() == 2 else torch.int32)
    bi = b.contiguous().view(torch.int16 if b.element_size() == 2 else torch.int32)
    n = int((ai != bi).sum())
    assert n == 0, f"{name}: {n} of {ai.numel()} elements differ"


def _both(c, inp):
    q, k, v, dout = (inp[x].to(DEV) for x in ("q", "k", "v", "dout"))
    pr, st = lh.attention_forward(q, k, v, c.p, c.L, c.k, flags=c.flags)
    grads = lh.attention_backward(pr, st, dout)
    pri, sti = lh.attention_forward_indexed(q, k, v, c.p, c.L, c.k, flags=c.flags)
    gradsi = lh.attention_backward_indexed(pri, q, k, v, sti, dout)
    torch.cuda.synchronize()
    return (st, grads), (sti, gradsi)


@pytest.mark.parametrize("name", ["t_gqa", "t_p3", "t_l1", "t_k0", "t_strat", "t_l2", "t_g3", "c2"])
def test_indexed_layer_is_bitwise_the_materialised_layer(name):
    c = _cfg(name)
    print(f"[indexed] {name}", flush=True)
    inp = workloads.make_inputs(c)
    (st, (dq, dk, dv)), (sti, (dqi, dki, dvi)) = _both(c, inp)
    for key in ("idx", "slot", "os", "lse", "o"):
        _same(key, sti[key], st[key])
    _same("dq", dqi, dq)
    _same("dk", dki, dk)
    _same("dv", dvi, dv)


@pytest.mark.parametrize("name", ["t_gqa", "t_p3", "t_strat", "t_g3"])
def test_indexed_layer_matches_oracle(name):
    """The indexed layer's own outputs (forward and backward) against the oracle, at the same
    bar as the materialised layer."""
    c = _cfg(name)
    print(f"[indexed vs oracle] {name}", flush=True)
    inp = workloads.make_inputs(c)
    q, k, v, dout = (inp[x].to(DEV) for x in ("q", "k", "v", "dout"))
    pri, sti = lh.attention_forward_indexed(q, k, v, c.p, c.L, c.k, flags=c.flags)
    grads = lh.attention_backward_indexed(pri, q, k, v, sti, dout)
    torch.cuda.synchronize()
    check_layer(c, inp, sti, grads)


def test_indexed_stage_calls_match_gathered_rows():
    """lh_sdpa_fwd_indexed / lh_sdpa_bwd_indexed against lh_sdpa_fwd / lh_sdpa_bwd on the rows
    lh_gather materialises, and against the oracle."""
    c = _cfg("t_gqa")
    inp = workloads.make_inputs(c)
    q, k, v, dout = (inp[x].to(DEV) for x in ("q", "k", "v", "dout"))
    pr, st = lh.attention_forward(q, k, v, c.p, c.L, c.k)
    S, Ptot = lh.lh_subseq_len(pr), lh.lh_pyramid_rows(pr)
    R = Ptot - c.N
    qp = torch.empty(c.B, R, c.Hq, c.D, dtype=q.dtype, device=DEV)
    kp = torch.empty(c.B, R, c.Hkv, c.D, dtype=q.dtype, device=DEV)
    vp = torch.empty_like(kp)
    lh.lh_pyramid_pool(pr, q, k, v, qp, kp, vp)
    os_, lse = torch.empty_like(st["os"]), torch.empty_like(st["lse"])
    lh.lh_sdpa_fwd_indexed(pr, q, k, v, qp, kp, vp, st["idx"], os_, lse)
    torch.cuda.synchronize()
    _same("os", os_, st["os"])
    _same("lse", lse, st["lse"])
    dos = torch.randn(st["os"].shape, generator=torch.Generator().manual_seed(5)).to(q.dtype).to(DEV)
    ws = lh.workspace(pr, lh.LH_OP_SDPA_BWD)
    ref = [torch.empty_like(st["qs"]) for _ in range(3)]
    got = [torch.empty_like(st["qs"]) for _ in range(3)]
    lh.lh_sdpa_bwd(pr, st["qs"], st["ks"], st["vs"], st["os"], st["lse"], dos, *ref, ws)
    lh.lh_sdpa_bwd_indexed(pr, q, k, v, qp, kp, vp, st["idx"], st["os"], st["lse"], dos, *got, ws)
    torch.cuda.synchronize()
    for nm, a, b in zip(("dqs", "dks", "dvs"), got, ref):
        _same(nm, a, b)
    # and the oracle, through the layer
    qn, kn, vn = (inp[x].double().numpy() for x in ("q", "k", "v"))
    f = oracle.layer_forward(qn, kn, vn, c.p, c.L, c.k, dtype=oracle.BF16)
    check_equal("idx", st["idx"], f["idx"])
    check_close_heads("os", os_, f["os"], c.dtype, 1)


def test_indexed_layer_full_size_c4():
    """The benchmark workload: the indexed layer gives the same bits as the materialised one."""
    c = workloads.CONFIGS["c4"]
    print("[indexed] c4", flush=True)
    inp = workloads.make_inputs(c, device=DEV)
    q, k, v, dout = inp["q"], inp["k"], inp["v"], inp["dout"]
    pr, st = lh.attention_forward(q, k, v, c.p, c.L, c.k)
    dq, dk, dv = lh.attention_backward(pr, st, dout)
    keep = {x: st[x] for x in ("idx", "slot", "os", "lse", "o")}
    del st
    pri, sti = lh.attention_forward_indexed(q, k, v, c.p, c.L, c.k)
    dqi, dki, dvi = lh.attention_backward_indexed(pri, q, k, v, sti, dout)
    torch.cuda.synchronize()
    for key in keep:
        _same(key, sti[key], keep[key])
    _same("dq", dqi, dq)
    _same("dk", dki, dk)
    _same("dv", dvi, dv)
