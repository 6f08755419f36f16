"""The fused layer under HIP graph capture. lh_attention_fwd and lh_attention_bwd only enqueue
kernels on the caller's stream (no allocation, memset or host synchronization), so one forward
and one backward call can be captured into a graph and replayed. The replays run with eager work
and synchronizations between them, and every replay is compared bit for bit with eager calls on
the same inputs, including replays after the inputs were overwritten in place."""
import pytest
import torch

import workloads

lh = pytest.importorskip("paper_2605_06554_amd")

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _buffers(pr, q, k):
    B, N, Hq, D = q.shape
    S, Ptot = lh.lh_subseq_len(pr), lh.lh_pyramid_rows(pr)
    Hs = lh.selection_heads(pr)
    e = lambda *s, dt=q.dtype: torch.empty(*s, dtype=dt, device=DEV)
    return dict(
        o=torch.empty_like(q), idx=e(B, Hs, S, dt=torch.int32), slot=e(B, Hs, Ptot, dt=torch.int32),
        qs=e(B, Hq, S, D), ks=e(B, Hs, S, D), vs=e(B, Hs, S, D), os=e(B, Hq, S, D),
        lse=e(B, Hq, S, dt=torch.float32), dq=torch.empty_like(q), dk=torch.empty_like(k), dv=torch.empty_like(k),
        wsf=lh.workspace(pr, lh.LH_OP_ATTENTION_FWD), wsb=lh.workspace(pr, lh.LH_OP_ATTENTION_BWD))


def _layer(pr, x, b):
    q, k, v, dout = x
    lh.lh_attention_fwd(pr, q, k, v, b["o"], b["idx"], b["slot"], b["qs"], b["ks"], b["vs"], b["os"], b["lse"],
                        b["wsf"])
    lh.lh_attention_bwd(pr, b["idx"], b["slot"], b["qs"], b["ks"], b["vs"], b["os"], b["lse"], dout, b["dq"],
                        b["dk"], b["dv"], b["wsb"])


KEYS = ("o", "idx", "slot", "os", "lse", "dq", "dk", "dv")


@pytest.mark.parametrize("name", ["t_gqa", "t_gqs"])
def test_layer_graph_replays_match_eager(name):
    c = workloads.TEST_CONFIGS[name]
    print(f"[graph] {name}", flush=True)
    sets = []
    for seed in (c.seed, c.seed + 1):
        inp = workloads.make_inputs(workloads.scaled(c, seed=seed))
        sets.append(tuple(inp[x].to(DEV) for x in ("q", "k", "v", "dout")))
    q0, k0 = sets[0][0], sets[0][1]
    B, N, Hq, D = q0.shape
    pr = lh.problem(B, N, Hq, k0.shape[2], D, c.p, c.L, c.k, q0.dtype, flags=c.flags)
    assert lh.lh_check(pr) == lh.LH_OK

    # eager reference of each input set, in buffers of its own
    ref = []
    for x in sets:
        b = _buffers(pr, q0, k0)
        _layer(pr, x, b)
        torch.cuda.synchronize()
        ref.append({key: b[key].clone() for key in KEYS})

    # graph over fixed input and output buffers; warm up on the capture stream first
    xin = tuple(t.clone() for t in sets[0])
    b = _buffers(pr, q0, k0)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        _layer(pr, xin, b)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        _layer(pr, xin, b)
    torch.cuda.synchronize()

    for rep, which in enumerate((0, 0, 1, 0, 1)):
        for t, src in zip(xin, sets[which]):
            t.copy_(src)  # eager work between replays: new inputs in place, outputs poisoned
        for key in KEYS:
            b[key].fill_(-7 if b[key].dtype == torch.int32 else float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for key in KEYS:
            assert torch.equal(b[key], ref[which][key]), f"replay {rep} (inputs {which}): {key}"
