"""The GQA-shared selection mode (LH_FLAG_GQA_SHARED) against the oracle: one selection per KV
group, per-group idx / slot / ks / vs, per-query-head qs / os / lse / o and gradients."""
import numpy as np
import pytest
import torch

import oracle
import workloads
from parity import check_equal, check_layer

lh = pytest.importorskip("paper_2605_06554_amd")

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.mark.parametrize("name", ["t_gqs", "t_gqs3", "t_gqs_f32"])
def test_shared_layer_matches_oracle(name):
    c = workloads.TEST_CONFIGS[name]
    print(f"[gqa-shared] {name}", flush=True)
    inp = workloads.make_inputs(c)
    q, k, v, dout = (inp[x].to(DEV) for x in ("q", "k", "v", "dout"))
    pr, st = lh.attention_forward(q, k, v, c.p, c.L, c.k, flags=c.flags)
    dq, dk, dv = lh.attention_backward(pr, st, dout)
    torch.cuda.synchronize()
    assert st["idx"].shape[1] == c.Hkv and st["ks"].shape[1] == c.Hkv
    check_layer(c, inp, st, (dq, dk, dv))


def test_shared_indexed_layer_is_bitwise_the_materialised_layer():
    c = workloads.TEST_CONFIGS["t_gqs"]
    inp = workloads.make_inputs(c)
    q, k, v, dout = (inp[x].to(DEV) for x in ("q", "k", "v", "dout"))
    pr, st = lh.attention_forward(q, k, v, c.p, c.L, c.k, flags=c.flags)
    grads = lh.attention_backward(pr, st, dout)
    pri, sti = lh.attention_forward_indexed(q, k, v, c.p, c.L, c.k, flags=c.flags)
    gradsi = lh.attention_backward_indexed(pri, q, k, v, sti, dout)
    torch.cuda.synchronize()
    for key in ("idx", "slot", "os", "lse", "o"):
        assert torch.equal(sti[key], st[key]), key
    for nm, a, b in zip(("dq", "dk", "dv"), gradsi, grads):
        assert torch.equal(a, b), nm


def test_shared_selection_at_c4_size():
    """The benchmark shapes with one selection per KV group: the scores, selection and gathered
    rows of KV groups 0 and 7 bit for bit (the oracle computes them in full)."""
    c = workloads.scaled(workloads.CONFIGS["c4"], flags=lh.LH_FLAG_GQA_SHARED)
    print("[gqa-shared] c4 size", flush=True)
    inp = workloads.make_inputs(c, device=DEV)
    q, k, v = inp["q"], inp["k"], inp["v"]
    pr, st = lh.attention_forward(q, k, v, c.p, c.L, c.k, flags=c.flags)
    torch.cuda.synchronize()
    G = c.Hq // c.Hkv
    h = oracle.Head(c.N, c.D, c.p, c.L, c.k, oracle.BF16)
    for gg in (0, c.Hkv - 1):
        host = lambda t: np.ascontiguousarray(t.double().cpu().numpy())
        kh = host(k[0, :, gg])
        s_qk = np.maximum.reduce([oracle.scores(h, host(q[0, :, gg * G + t])) for t in range(G)])
        idx, slot = oracle.select(h, s_qk, oracle.scores(h, kh))
        check_equal(f"idx[{gg}]", st["idx"][0, gg], idx)
        check_equal(f"slot[{gg}]", st["slot"][0, gg], slot)
        check_equal(f"ks[{gg}]", host(st["ks"][0, gg]), oracle.gather(h, oracle.pool(h, kh), idx))
        qh = host(q[0, :, gg * G + 1])
        check_equal(f"qs[{gg * G + 1}]", host(st["qs"][0, gg * G + 1]), oracle.gather(h, oracle.pool(h, qh), idx))
