"""lh_sdpa_bwd_noalloc (the SDPA backward with its Delta in the library's static device scratch)
against lh_sdpa_bwd with a caller workspace, through the C ABI: two calls in a row, the second
on a smaller problem, in bf16 and fp32; and the refusal of a problem larger than the scratch."""
import numpy as np
import pytest
import torch

lh = pytest.importorskip("paper_2605_06554_amd")

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _inputs(B, H, Hkv, S, D, dtype, seed):
    """L = 1: the SDPA runs on S rows. With Hkv < H the selection is shared per KV group, so
    K~ and V~ have Hkv heads (the grouped dK / dV path); otherwise every head has its own."""
    g = torch.Generator(DEV).manual_seed(seed)
    flags = lh.LH_FLAG_GQA_SHARED if Hkv < H else 0
    pr = lh.problem(B, S, H, Hkv, D, 2, 1, 0, dtype, 0.0, flags)
    assert lh.lh_subseq_len(pr) == S
    mk = lambda h: torch.randn(B, h, S, D, generator=g, device=DEV).to(dtype)
    qs, ks, vs = mk(H), mk(Hkv), mk(Hkv)
    os_ = torch.empty_like(qs)
    lse = torch.empty(B, H, S, dtype=torch.float32, device=DEV)
    lh.lh_sdpa_fwd(pr, qs, ks, vs, os_, lse)
    dos = mk(H)
    return pr, (qs, ks, vs, os_, lse, dos)


def _both(pr, x):
    qs, ks, vs = x[:3]
    ref = [torch.empty_like(qs), torch.empty_like(ks), torch.empty_like(vs)]
    got = [torch.full_like(t, 7.0) for t in ref]
    ws = lh.workspace(pr, lh.LH_OP_SDPA_BWD)
    lh.lh_sdpa_bwd(pr, *x, *ref, ws)
    lh.lh_sdpa_bwd_noalloc(pr, *x, *got)
    torch.cuda.synchronize()
    return ref, got


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_noalloc_matches_workspace_call_twice(dtype):
    # first a large problem (its Delta fills most of the 16 MiB scratch), then a smaller one
    shapes = [(1, 32, 8, 120000, 128), (2, 3, 3, 777, 64)] if dtype == torch.bfloat16 else \
             [(1, 8, 4, 3000, 128), (1, 2, 2, 257, 64)]
    for n, (B, H, Hkv, S, D) in enumerate(shapes):
        print(f"[noalloc] {dtype} call {n}: B={B} H={H} Hkv={Hkv} S={S} D={D}", flush=True)
        pr, x = _inputs(B, H, Hkv, S, D, dtype, 100 + n)
        ref, got = _both(pr, x)
        for name, a, b in zip(("dqs", "dks", "dvs"), got, ref):
            assert torch.equal(a, b), f"{name} differs from lh_sdpa_bwd (call {n})"


def test_noalloc_refuses_more_than_its_scratch():
    import ctypes

    pr = lh.problem(1, 65536, 65, 65, 128, 2, 1, 0, torch.bfloat16)  # B * Hq * S = 4,259,840 > 4,194,304
    assert lh.lh_check(pr) == lh.LH_OK
    dummy = torch.empty(16, dtype=torch.bfloat16, device=DEV)
    st = lh._load().lh_sdpa_bwd_noalloc(ctypes.byref(pr), *([dummy.data_ptr()] * 9), None)
    assert st == -6 and "static scratch" in lh.lh_last_error()
