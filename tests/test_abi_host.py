"""Host-only checks of the C ABI: the library loads, exports every declared entry point, and its
validation and shape math agree with the oracle (no device calls)."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
import workloads
import paper_2605_06554_amd as lh

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "lighthouse.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(lh_[a-z_0-9]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(lh.library_path)
    names = _declared()
    assert len(names) >= 19
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(lh.EXPORTED) == names


def _pr(**kw):
    base = dict(B=1, N=1024, Hq=2, Hkv=2, D=64, p=4, L=3, k=128, dtype=lh.LH_F32)
    base.update(kw)
    return lh.problem(**base)


@pytest.mark.parametrize("kw,code", [
    (dict(), 0),
    (dict(N=1000), -2),                 # 16 does not divide 1000
    (dict(p=1), -3),
    (dict(L=0), -3),
    (dict(L=9), -3),
    (dict(k=-1), -3),
    (dict(Hq=3, Hkv=2), -3),
    (dict(D=96), -3),
    (dict(dtype=7), -4),
    (dict(flags=8), -3),
    (dict(N=0), -2),
    (dict(L=1, p=0), 0),                # p is irrelevant with one level
    (dict(N=2 ** 20, L=2, k=1000), 0),   # a level of 262144 candidates ranks with its keys in the workspace
    (dict(N=2 ** 28, p=2, L=2, k=1), -3),  # 2^27 candidates at one level: beyond the 2^26 supported
    (dict(scale=-0.125), -3),           # a negative softmax scale is refused
    (dict(scale=float("nan")), -8),     # a non-finite scale: LH_E_NONFINITE
    (dict(scale=float("inf")), -8),
])
def test_check_codes(kw, code):
    pr = _pr(**kw)
    assert lh.lh_check(pr) == code
    if code != 0:
        assert lh.lh_last_error() != ""
        assert lh.lh_subseq_len(pr) == -1


def test_null_problem():
    lib = ctypes.CDLL(lh.library_path)
    lib.lh_check.argtypes = [ctypes.c_void_p]
    assert lib.lh_check(None) == -1


@pytest.mark.parametrize("name", list(workloads.CONFIGS) + list(workloads.TEST_CONFIGS))
def test_shapes_match_oracle(name, rng):
    c = {**workloads.CONFIGS, **workloads.TEST_CONFIGS}[name]
    pr = lh.problem(c.B, c.N, c.Hq, c.Hkv, c.D, c.p, c.L, c.k, lh.LH_BF16, 0.0, c.flags)
    assert lh.lh_check(pr) == 0
    h = oracle.Head(c.N, c.D, c.p, c.L, c.k, oracle.F32, c.flags)
    assert lh.lh_pyramid_rows(pr) == h.ptot
    for l in range(c.L):
        assert lh.lh_level_rows(pr, l) == h.level_rows(l)
        assert lh.lh_level_offset(pr, l) == h.level_offset(l)
    assert lh.lh_level_rows(pr, c.L) == -1
    if h.ptot <= 400000:
        s = rng.random(h.ptot).astype(np.float32)
        idx, _ = oracle.select(h, s, s)
        assert lh.lh_subseq_len(pr) == len(idx)


@pytest.mark.parametrize("flags", [0, lh.LH_FLAG_REPLACE_PARENTS, lh.LH_FLAG_STRATIFIED])
@pytest.mark.parametrize("N,p,L,k", [(64, 2, 4, 3), (256, 4, 4, 300), (81, 3, 3, 4), (777, 4, 1, 0)])
def test_subseq_len_matches_oracle_selection(N, p, L, k, flags, rng):
    pr = lh.problem(1, N, 1, 1, 64, p, L, k, lh.LH_F32, 0.0, flags)
    h = oracle.Head(N, 64, p, L, k, oracle.F32, flags)
    s = rng.random(h.ptot).astype(np.float32)
    idx, _ = oracle.select(h, s, s)
    assert lh.lh_subseq_len(pr) == len(idx)


def test_workspace_sizes():
    c = workloads.CONFIGS["c4"]
    pr = lh.problem(c.B, c.N, c.Hq, c.Hkv, c.D, c.p, c.L, c.k, lh.LH_BF16)
    S = lh.lh_subseq_len(pr)
    assert S == 54272
    assert lh.lh_workspace_bytes(pr, lh.LH_OP_SDPA_BWD) >= c.B * c.Hq * S * 4
    fwd = lh.lh_workspace_bytes(pr, lh.LH_OP_ATTENTION_FWD)
    R = lh.lh_pyramid_rows(pr) - c.N
    assert fwd >= (c.Hq + 2 * c.Hkv) * R * c.D * 2 + (c.Hq + c.Hkv) * lh.lh_pyramid_rows(pr) * 4
    assert lh.lh_workspace_bytes(pr, lh.LH_OP_ATTENTION_BWD) >= 4 * c.Hq * S * c.D * 2
    with pytest.raises(lh.LighthouseError):
        lh.lh_workspace_bytes(pr, 99)


def test_entry_points_reject_bad_pointers_before_any_launch():
    # argument errors are caught on the host: no device is touched
    pr = _pr()
    lib = ctypes.CDLL(lh.library_path)
    lib.lh_sdpa_fwd.argtypes = [ctypes.POINTER(lh.lh_problem)] + [ctypes.c_void_p] * 6
    assert lib.lh_sdpa_fwd(ctypes.byref(pr), None, None, None, None, None, None) == -1
    assert lib.lh_sdpa_fwd(ctypes.byref(pr), 0x1001, 0x2000, 0x3000, 0x4000, 0x5000, None) == -5
    lib.lh_select_topk.argtypes = [ctypes.POINTER(lh.lh_problem)] + [ctypes.c_void_p] * 5 + [ctypes.c_size_t, ctypes.c_void_p]
    assert lib.lh_select_topk(ctypes.byref(pr), 0x1000, 0x2000, 0x3000, 0x4000, None, 0, None) == -6
    assert lib.lh_select_topk(ctypes.byref(pr), 0x1000, 0x2000, 0x3000, 0x4000, 0x5000, 16, None) == -6
    bad = _pr(N=1000)
    assert lib.lh_sdpa_fwd(ctypes.byref(bad), 0x1000, 0x2000, 0x3000, 0x4000, 0x5000, None) == -2


def test_indexed_entry_points_are_bf16_only():
    """The index-driven SDPA is built for bf16: fp32 problems are rejected on the host, before
    any pointer is looked at or anything is launched."""
    pr = _pr(dtype=lh.LH_F32)
    lib = lh._load()
    z = None
    assert lib.lh_sdpa_fwd_indexed(ctypes.byref(pr), z, z, z, z, z, z, z, z, z, z) == -4
    assert "bf16" in lh.lh_last_error()
    assert lib.lh_sdpa_bwd_indexed(ctypes.byref(pr), *([z] * 14), 0, z) == -4
    assert lib.lh_attention_fwd_indexed(ctypes.byref(pr), *([z] * 12), 0, z) == -4
    assert lib.lh_attention_bwd_indexed(ctypes.byref(pr), *([z] * 15), 0, z) == -4
    # bf16 with a NULL input is a pointer error, still on the host
    pr16 = _pr(dtype=lh.LH_BF16)
    assert lib.lh_sdpa_fwd_indexed(ctypes.byref(pr16), z, z, z, z, z, z, z, z, z, z) == -1


def test_indexed_forward_workspace_is_the_scores_and_lists():
    """lh_attention_fwd_indexed keeps no pyramid in its workspace: it needs the forward
    workspace minus the three pyramid buffers."""
    pr = _pr(dtype=lh.LH_BF16, B=2, N=4096, Hq=4, Hkv=2, D=128, p=4, L=4, k=256)
    full = lh.lh_workspace_bytes(pr, lh.LH_OP_ATTENTION_FWD)
    idx = lh.lh_workspace_bytes(pr, lh.LH_OP_ATTENTION_FWD_INDEXED)
    R = lh.lh_pyramid_rows(pr) - 4096
    al = lambda n: (n + 255) // 256 * 256
    assert full - idx == al(2 * R * 4 * 128 * 2) + 2 * al(2 * R * 2 * 128 * 2)


class _FakeDeviceTensor:
    """Stands in for a device tensor on a host without a GPU (only what the binding reads)."""

    def __init__(self, n, dtype, contiguous=True):
        self.n, self.dtype, self.contiguous, self.is_cuda = n, dtype, contiguous, True

    def numel(self):
        return self.n

    def is_contiguous(self):
        return self.contiguous


def test_binding_refuses_bad_tensors_before_the_library():
    """The Python binding checks device, layout, dtype and size of every tensor against the
    problem before passing its address on: a short buffer would otherwise be read or written
    past its end by a kernel."""
    import torch
    pr = _pr(dtype=lh.LH_BF16, B=1, N=1024, Hq=2, Hkv=1, D=64, p=4, L=3, k=16)
    S = lh.lh_subseq_len(pr)
    n_qs, n_kvs, n_lse = 2 * S * 64, 2 * S * 64, 2 * S  # selection heads = Hq = 2
    good = lambda n, dt=torch.bfloat16: _FakeDeviceTensor(n, dt)
    ok = (good(n_qs), good(n_kvs), good(n_kvs), good(n_qs), good(n_lse, torch.float32))
    cases = [
        ((torch.zeros(4),) + ok[1:], "not a device tensor"),
        ((_FakeDeviceTensor(n_qs, torch.bfloat16, False),) + ok[1:], "not contiguous"),
        ((good(n_qs, torch.float32),) + ok[1:], "dtype"),
        (ok[:1] + (good(n_kvs - 1),) + ok[2:], "elements"),
        (ok[:4] + (good(n_lse - 1, torch.float32),), "elements"),
    ]
    for args, msg in cases:
        with pytest.raises(lh.LighthouseError, match=msg):
            lh.lh_sdpa_fwd(pr, *args)
    # with GQA-shared selection, ks and vs hold one row block per KV head
    prs = _pr(dtype=lh.LH_BF16, B=1, N=1024, Hq=2, Hkv=1, D=64, p=4, L=3, k=16, flags=lh.LH_FLAG_GQA_SHARED)
    Ss = lh.lh_subseq_len(prs)
    with pytest.raises(lh.LighthouseError, match="ks has"):
        lh.lh_sdpa_fwd(prs, good(2 * Ss * 64), good(Ss * 64 - 1), good(Ss * 64), good(2 * Ss * 64),
                       good(2 * Ss, torch.float32))
