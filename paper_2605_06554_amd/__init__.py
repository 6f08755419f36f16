"""Lighthouse attention hot path on AMD MI355X (gfx950): Python binding of liblighthouse.so.

The binding only marshals arguments: torch tensors supply device memory and the current HIP
stream; every step of the layer runs in the library's HIP kernels. Each ``lh_*`` function has
the same name and argument order as its C declaration in ``include/lighthouse.h`` and raises
``LighthouseError`` on a non-OK status. There is no fallback: if the library is missing or a
call fails, the error is raised.
"""
from __future__ import annotations

import ctypes
import os

import torch

__all__ = [
    "LH_OK", "LH_F32", "LH_BF16", "LH_FLAG_REPLACE_PARENTS", "LH_FLAG_STRATIFIED", "LH_FLAG_GQA_SHARED", "LH_OP_SELECT", "LH_OP_SDPA_BWD",
    "LH_OP_ATTENTION_FWD", "LH_OP_ATTENTION_BWD", "LH_OP_ATTENTION_FWD_INDEXED", "LighthouseError", "lh_problem", "problem",
    "lh_check", "lh_level_rows", "lh_level_offset", "lh_pyramid_rows", "lh_subseq_len",
    "lh_workspace_bytes", "lh_status_str", "lh_last_error", "lh_pyramid_pool", "lh_score",
    "lh_pool_score", "lh_select_topk", "lh_gather", "lh_sdpa_fwd", "lh_sdpa_bwd", "lh_scatter",
    "lh_scatter_bwd", "lh_gather_bwd", "lh_attention_fwd", "lh_attention_bwd", "lh_sdpa_fwd_indexed",
    "lh_sdpa_bwd_indexed", "lh_attention_fwd_indexed", "lh_attention_bwd_indexed", "workspace",
    "attention_forward", "attention_backward", "attention_forward_indexed", "attention_backward_indexed",
    "selection_heads",
    "library_path", "EXPORTED",
]

LH_OK = 0
LH_F32, LH_BF16 = 0, 1
LH_FLAG_REPLACE_PARENTS = 1
LH_FLAG_STRATIFIED = 2
LH_FLAG_GQA_SHARED = 4
LH_OP_SELECT, LH_OP_SDPA_BWD, LH_OP_ATTENTION_FWD, LH_OP_ATTENTION_BWD, LH_OP_ATTENTION_FWD_INDEXED = 0, 1, 2, 3, 4

_HERE = os.path.dirname(os.path.abspath(__file__))
library_path = os.path.join(_HERE, "liblighthouse.so")

EXPORTED = [
    "lh_check", "lh_level_rows", "lh_level_offset", "lh_pyramid_rows", "lh_subseq_len",
    "lh_workspace_bytes", "lh_status_str", "lh_last_error", "lh_pyramid_pool", "lh_score",
    "lh_pool_score", "lh_select_topk", "lh_gather", "lh_sdpa_fwd", "lh_sdpa_bwd", "lh_sdpa_bwd_noalloc",
    "lh_scatter", "lh_scatter_bwd",
    "lh_gather_bwd", "lh_attention_fwd", "lh_attention_bwd", "lh_sdpa_fwd_indexed", "lh_sdpa_bwd_indexed",
    "lh_attention_fwd_indexed", "lh_attention_bwd_indexed",
]


class LighthouseError(RuntimeError):
    pass


class lh_problem(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int64), ("N", ctypes.c_int64), ("Hq", ctypes.c_int32),
                ("Hkv", ctypes.c_int32), ("D", ctypes.c_int32), ("p", ctypes.c_int32),
                ("L", ctypes.c_int32), ("k", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("scale", ctypes.c_float), ("flags", ctypes.c_uint32)]

    def __repr__(self):
        return ("lh_problem(B=%d, N=%d, Hq=%d, Hkv=%d, D=%d, p=%d, L=%d, k=%d, dtype=%d, scale=%g, flags=%d)"
                % (self.B, self.N, self.Hq, self.Hkv, self.D, self.p, self.L, self.k, self.dtype,
                   self.scale, self.flags))


def problem(B, N, Hq, Hkv, D, p, L, k, dtype=LH_BF16, scale=0.0, flags=0) -> lh_problem:
    if isinstance(dtype, torch.dtype):
        dtype = {torch.float32: LH_F32, torch.bfloat16: LH_BF16}[dtype]
    return lh_problem(B, N, Hq, Hkv, D, p, L, k, dtype, scale, flags)


_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(library_path):
        raise LighthouseError(
            f"{library_path} is not built; build it with `python -m paper_2605_06554_amd.build`")
    lib = ctypes.CDLL(library_path)
    P, PR = ctypes.c_void_p, ctypes.POINTER(lh_problem)
    i32, i64, sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    sigs = {
        "lh_check": (i32, [PR]),
        "lh_level_rows": (i64, [PR, i32]),
        "lh_level_offset": (i64, [PR, i32]),
        "lh_pyramid_rows": (i64, [PR]),
        "lh_subseq_len": (i64, [PR]),
        "lh_workspace_bytes": (i32, [PR, i32, ctypes.POINTER(sz)]),
        "lh_status_str": (ctypes.c_char_p, [i32]),
        "lh_last_error": (ctypes.c_char_p, []),
        "lh_pyramid_pool": (i32, [PR, P, P, P, P, P, P, P]),
        "lh_score": (i32, [PR, P, P, P, P, P]),
        "lh_pool_score": (i32, [PR, P, P, P, P, P, P, P, P, P]),
        "lh_select_topk": (i32, [PR, P, P, P, P, P, sz, P]),
        "lh_gather": (i32, [PR, P, P, P, P, P, P, P, P, P, P, P]),
        "lh_sdpa_fwd": (i32, [PR, P, P, P, P, P, P]),
        "lh_sdpa_bwd": (i32, [PR, P, P, P, P, P, P, P, P, P, P, sz, P]),
        "lh_sdpa_bwd_noalloc": (i32, [PR, P, P, P, P, P, P, P, P, P, P]),
        "lh_scatter": (i32, [PR, P, P, P, P]),
        "lh_scatter_bwd": (i32, [PR, P, P, P, P]),
        "lh_gather_bwd": (i32, [PR, P, P, P, P, P, P, P, P]),
        "lh_attention_fwd": (i32, [PR, P, P, P, P, P, P, P, P, P, P, P, P, sz, P]),
        "lh_attention_bwd": (i32, [PR, P, P, P, P, P, P, P, P, P, P, P, P, sz, P]),
        "lh_sdpa_fwd_indexed": (i32, [PR, P, P, P, P, P, P, P, P, P, P]),
        "lh_sdpa_bwd_indexed": (i32, [PR, P, P, P, P, P, P, P, P, P, P, P, P, P, P, sz, P]),
        "lh_attention_fwd_indexed": (i32, [PR, P, P, P, P, P, P, P, P, P, P, P, P, sz, P]),
        "lh_attention_bwd_indexed": (i32, [PR, P, P, P, P, P, P, P, P, P, P, P, P, P, P, P, sz, P]),
    }
    for name, (res, args) in sigs.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


def _p(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _nbytes(t):
    return 0 if t is None else t.numel() * t.element_size()


def _call(name, *args):
    st = getattr(_load(), name)(*args)
    if st != LH_OK:
        raise LighthouseError(f"{name}: {lh_status_str(st)}: {lh_last_error()}")


# ---------------------------------------------------------------- host-only helpers

def lh_check(pr: lh_problem) -> int:
    return _load().lh_check(ctypes.byref(pr))


def lh_level_rows(pr, level):
    return _load().lh_level_rows(ctypes.byref(pr), level)


def lh_level_offset(pr, level):
    return _load().lh_level_offset(ctypes.byref(pr), level)


def lh_pyramid_rows(pr):
    return _load().lh_pyramid_rows(ctypes.byref(pr))


def lh_subseq_len(pr):
    return _load().lh_subseq_len(ctypes.byref(pr))


def lh_workspace_bytes(pr, op) -> int:
    out = ctypes.c_size_t(0)
    _call("lh_workspace_bytes", ctypes.byref(pr), op, ctypes.byref(out))
    return out.value


def lh_status_str(st) -> str:
    return _load().lh_status_str(st).decode()


def lh_last_error() -> str:
    return _load().lh_last_error().decode()


# ---------------------------------------------------------------- tensor checks
# A kernel trusts the sizes the problem implies, so a torch tensor that is too small, strided,
# on the host or of another dtype is refused here, before its address reaches the library.
# Raw integer addresses and None are passed through unchecked (the library rejects NULL).

class _Sizes:
    def __init__(self, pr, S, Ptot):
        self.B, self.N, self.Hq, self.Hkv, self.D = pr.B, pr.N, pr.Hq, pr.Hkv, pr.D
        self.S, self.Ptot, self.R, self.Hs = S, Ptot, Ptot - pr.N, selection_heads(pr)


_KINDS = {  # element count from the problem's sizes, dtype (None: the problem's)
    "q": (lambda z: z.B * z.N * z.Hq * z.D, None),
    "kv": (lambda z: z.B * z.N * z.Hkv * z.D, None),
    "qpyr": (lambda z: z.B * z.R * z.Hq * z.D, None),
    "kvpyr": (lambda z: z.B * z.R * z.Hkv * z.D, None),
    "s_qk": (lambda z: z.B * z.Hq * z.Ptot, torch.float32),
    "s_kq": (lambda z: z.B * z.Hkv * z.Ptot, torch.float32),
    "idx": (lambda z: z.B * z.Hs * z.S, torch.int32),
    "slot": (lambda z: z.B * z.Hs * z.Ptot, torch.int32),
    "qs": (lambda z: z.B * z.Hq * z.S * z.D, None),
    "kvs": (lambda z: z.B * z.Hs * z.S * z.D, None),
    "lse": (lambda z: z.B * z.Hq * z.S, torch.float32),
    "ws": (lambda z: 0, torch.uint8),
}


def _need(fn, pr, *args):
    """args: (tensor, argument name, kind) triples for the buffers of entry point fn."""
    S, Ptot = lh_subseq_len(pr), lh_pyramid_rows(pr)
    if S < 0 or Ptot < 0:
        return  # an invalid problem: the library's own check reports it
    z = _Sizes(pr, S, Ptot)
    xdt = torch.bfloat16 if pr.dtype == LH_BF16 else torch.float32
    for t, name, kind in args:
        if t is None or isinstance(t, int):
            continue
        count, dt = _KINDS[kind]
        dt = xdt if dt is None else dt
        n = count(z)
        if not t.is_cuda:
            raise LighthouseError(f"{fn}: {name} is not a device tensor")
        if not t.is_contiguous():
            raise LighthouseError(f"{fn}: {name} is not contiguous")
        if t.dtype != dt:
            raise LighthouseError(f"{fn}: {name} has dtype {t.dtype}, {dt} expected")
        if t.numel() < n:
            raise LighthouseError(f"{fn}: {name} has {t.numel()} elements, {n} needed")


# ---------------------------------------------------------------- stage entry points

def lh_pyramid_pool(pr, q, k, v, qpyr, kpyr, vpyr, stream=None):
    _need("lh_pyramid_pool", pr, (q, "q", "q"), (k, "k", "kv"), (v, "v", "kv"), (qpyr, "qpyr", "qpyr"),
          (kpyr, "kpyr", "kvpyr"), (vpyr, "vpyr", "kvpyr"))
    _call("lh_pyramid_pool", ctypes.byref(pr), _p(q), _p(k), _p(v), _p(qpyr), _p(kpyr), _p(vpyr), _stream(stream))


def lh_score(pr, q, k, s_qk, s_kq, stream=None):
    _need("lh_score", pr, (q, "q", "q"), (k, "k", "kv"), (s_qk, "s_qk", "s_qk"), (s_kq, "s_kq", "s_kq"))
    _call("lh_score", ctypes.byref(pr), _p(q), _p(k), _p(s_qk), _p(s_kq), _stream(stream))


def lh_pool_score(pr, q, k, v, qpyr, kpyr, vpyr, s_qk, s_kq, stream=None):
    _need("lh_pool_score", pr, (q, "q", "q"), (k, "k", "kv"), (v, "v", "kv"), (qpyr, "qpyr", "qpyr"),
          (kpyr, "kpyr", "kvpyr"), (vpyr, "vpyr", "kvpyr"), (s_qk, "s_qk", "s_qk"), (s_kq, "s_kq", "s_kq"))
    _call("lh_pool_score", ctypes.byref(pr), _p(q), _p(k), _p(v), _p(qpyr), _p(kpyr), _p(vpyr), _p(s_qk),
          _p(s_kq), _stream(stream))


def lh_select_topk(pr, s_qk, s_kq, idx, slot, ws, ws_bytes=None, stream=None):
    _need("lh_select_topk", pr, (s_qk, "s_qk", "s_qk"), (s_kq, "s_kq", "s_kq"), (idx, "idx", "idx"),
          (slot, "slot", "slot"), (ws, "ws", "ws"))
    _call("lh_select_topk", ctypes.byref(pr), _p(s_qk), _p(s_kq), _p(idx), _p(slot), _p(ws),
          _nbytes(ws) if ws_bytes is None else ws_bytes, _stream(stream))


def lh_gather(pr, q, k, v, qpyr, kpyr, vpyr, idx, qs, ks, vs, stream=None):
    _need("lh_gather", pr, (q, "q", "q"), (k, "k", "kv"), (v, "v", "kv"), (qpyr, "qpyr", "qpyr"),
          (kpyr, "kpyr", "kvpyr"), (vpyr, "vpyr", "kvpyr"), (idx, "idx", "idx"), (qs, "qs", "qs"),
          (ks, "ks", "kvs"), (vs, "vs", "kvs"))
    _call("lh_gather", ctypes.byref(pr), _p(q), _p(k), _p(v), _p(qpyr), _p(kpyr), _p(vpyr), _p(idx),
          _p(qs), _p(ks), _p(vs), _stream(stream))


def lh_sdpa_fwd(pr, qs, ks, vs, os_, lse, stream=None):
    _need("lh_sdpa_fwd", pr, (qs, "qs", "qs"), (ks, "ks", "kvs"), (vs, "vs", "kvs"), (os_, "os", "qs"),
          (lse, "lse", "lse"))
    _call("lh_sdpa_fwd", ctypes.byref(pr), _p(qs), _p(ks), _p(vs), _p(os_), _p(lse), _stream(stream))


def lh_sdpa_bwd(pr, qs, ks, vs, os_, lse, dos, dqs, dks, dvs, ws, ws_bytes=None, stream=None):
    _need("lh_sdpa_bwd", pr, (qs, "qs", "qs"), (ks, "ks", "kvs"), (vs, "vs", "kvs"), (os_, "os", "qs"),
          (lse, "lse", "lse"), (dos, "dos", "qs"), (dqs, "dqs", "qs"), (dks, "dks", "kvs"), (dvs, "dvs", "kvs"),
          (ws, "ws", "ws"))
    _call("lh_sdpa_bwd", ctypes.byref(pr), _p(qs), _p(ks), _p(vs), _p(os_), _p(lse), _p(dos), _p(dqs),
          _p(dks), _p(dvs), _p(ws), _nbytes(ws) if ws_bytes is None else ws_bytes, _stream(stream))


def lh_sdpa_bwd_noalloc(pr, qs, ks, vs, os_, lse, dos, dqs, dks, dvs, stream=None):
    """lh_sdpa_bwd with its workspace in the library's static device scratch (allocates nothing)."""
    _need("lh_sdpa_bwd_noalloc", pr, (qs, "qs", "qs"), (ks, "ks", "kvs"), (vs, "vs", "kvs"), (os_, "os", "qs"),
          (lse, "lse", "lse"), (dos, "dos", "qs"), (dqs, "dqs", "qs"), (dks, "dks", "kvs"), (dvs, "dvs", "kvs"))
    _call("lh_sdpa_bwd_noalloc", ctypes.byref(pr), _p(qs), _p(ks), _p(vs), _p(os_), _p(lse), _p(dos), _p(dqs),
          _p(dks), _p(dvs), _stream(stream))


def lh_scatter(pr, os_, slot, o, stream=None):
    _need("lh_scatter", pr, (os_, "os", "qs"), (slot, "slot", "slot"), (o, "o", "q"))
    _call("lh_scatter", ctypes.byref(pr), _p(os_), _p(slot), _p(o), _stream(stream))


def lh_scatter_bwd(pr, dout, slot, dos, stream=None):
    _need("lh_scatter_bwd", pr, (dout, "dout", "q"), (slot, "slot", "slot"), (dos, "dos", "qs"))
    _call("lh_scatter_bwd", ctypes.byref(pr), _p(dout), _p(slot), _p(dos), _stream(stream))


def lh_gather_bwd(pr, dqs, dks, dvs, slot, dq, dk, dv, stream=None):
    _need("lh_gather_bwd", pr, (dqs, "dqs", "qs"), (dks, "dks", "kvs"), (dvs, "dvs", "kvs"),
          (slot, "slot", "slot"), (dq, "dq", "q"), (dk, "dk", "kv"), (dv, "dv", "kv"))
    _call("lh_gather_bwd", ctypes.byref(pr), _p(dqs), _p(dks), _p(dvs), _p(slot), _p(dq), _p(dk), _p(dv),
          _stream(stream))


def lh_attention_fwd(pr, q, k, v, o, idx, slot, qs, ks, vs, os_, lse, ws, ws_bytes=None, stream=None):
    _need("lh_attention_fwd", pr, (q, "q", "q"), (k, "k", "kv"), (v, "v", "kv"), (o, "o", "q"),
          (idx, "idx", "idx"), (slot, "slot", "slot"), (qs, "qs", "qs"), (ks, "ks", "kvs"), (vs, "vs", "kvs"),
          (os_, "os", "qs"), (lse, "lse", "lse"), (ws, "ws", "ws"))
    _call("lh_attention_fwd", ctypes.byref(pr), _p(q), _p(k), _p(v), _p(o), _p(idx), _p(slot), _p(qs), _p(ks),
          _p(vs), _p(os_), _p(lse), _p(ws), _nbytes(ws) if ws_bytes is None else ws_bytes, _stream(stream))


def lh_attention_bwd(pr, idx, slot, qs, ks, vs, os_, lse, dout, dq, dk, dv, ws, ws_bytes=None, stream=None):
    _need("lh_attention_bwd", pr, (idx, "idx", "idx"), (slot, "slot", "slot"), (qs, "qs", "qs"),
          (ks, "ks", "kvs"), (vs, "vs", "kvs"), (os_, "os", "qs"), (lse, "lse", "lse"), (dout, "dout", "q"),
          (dq, "dq", "q"), (dk, "dk", "kv"), (dv, "dv", "kv"), (ws, "ws", "ws"))
    _call("lh_attention_bwd", ctypes.byref(pr), _p(idx), _p(slot), _p(qs), _p(ks), _p(vs), _p(os_), _p(lse),
          _p(dout), _p(dq), _p(dk), _p(dv), _p(ws), _nbytes(ws) if ws_bytes is None else ws_bytes,
          _stream(stream))


def lh_sdpa_fwd_indexed(pr, q, k, v, qpyr, kpyr, vpyr, idx, os_, lse, stream=None):
    _need("lh_sdpa_fwd_indexed", pr, (q, "q", "q"), (k, "k", "kv"), (v, "v", "kv"), (qpyr, "qpyr", "qpyr"),
          (kpyr, "kpyr", "kvpyr"), (vpyr, "vpyr", "kvpyr"), (idx, "idx", "idx"), (os_, "os", "qs"),
          (lse, "lse", "lse"))
    _call("lh_sdpa_fwd_indexed", ctypes.byref(pr), _p(q), _p(k), _p(v), _p(qpyr), _p(kpyr), _p(vpyr), _p(idx),
          _p(os_), _p(lse), _stream(stream))


def lh_sdpa_bwd_indexed(pr, q, k, v, qpyr, kpyr, vpyr, idx, os_, lse, dos, dqs, dks, dvs, ws, ws_bytes=None,
                        stream=None):
    _need("lh_sdpa_bwd_indexed", pr, (q, "q", "q"), (k, "k", "kv"), (v, "v", "kv"), (qpyr, "qpyr", "qpyr"),
          (kpyr, "kpyr", "kvpyr"), (vpyr, "vpyr", "kvpyr"), (idx, "idx", "idx"), (os_, "os", "qs"),
          (lse, "lse", "lse"), (dos, "dos", "qs"), (dqs, "dqs", "qs"), (dks, "dks", "kvs"), (dvs, "dvs", "kvs"),
          (ws, "ws", "ws"))
    _call("lh_sdpa_bwd_indexed", ctypes.byref(pr), _p(q), _p(k), _p(v), _p(qpyr), _p(kpyr), _p(vpyr), _p(idx),
          _p(os_), _p(lse), _p(dos), _p(dqs), _p(dks), _p(dvs), _p(ws),
          _nbytes(ws) if ws_bytes is None else ws_bytes, _stream(stream))


def lh_attention_fwd_indexed(pr, q, k, v, o, idx, slot, qpyr, kpyr, vpyr, os_, lse, ws, ws_bytes=None,
                             stream=None):
    _need("lh_attention_fwd_indexed", pr, (q, "q", "q"), (k, "k", "kv"), (v, "v", "kv"), (o, "o", "q"),
          (idx, "idx", "idx"), (slot, "slot", "slot"), (qpyr, "qpyr", "qpyr"), (kpyr, "kpyr", "kvpyr"),
          (vpyr, "vpyr", "kvpyr"), (os_, "os", "qs"), (lse, "lse", "lse"), (ws, "ws", "ws"))
    _call("lh_attention_fwd_indexed", ctypes.byref(pr), _p(q), _p(k), _p(v), _p(o), _p(idx), _p(slot),
          _p(qpyr), _p(kpyr), _p(vpyr), _p(os_), _p(lse), _p(ws), _nbytes(ws) if ws_bytes is None else ws_bytes,
          _stream(stream))


def lh_attention_bwd_indexed(pr, q, k, v, qpyr, kpyr, vpyr, idx, slot, os_, lse, dout, dq, dk, dv, ws,
                             ws_bytes=None, stream=None):
    _need("lh_attention_bwd_indexed", pr, (q, "q", "q"), (k, "k", "kv"), (v, "v", "kv"),
          (qpyr, "qpyr", "qpyr"), (kpyr, "kpyr", "kvpyr"), (vpyr, "vpyr", "kvpyr"), (idx, "idx", "idx"),
          (slot, "slot", "slot"), (os_, "os", "qs"), (lse, "lse", "lse"), (dout, "dout", "q"), (dq, "dq", "q"),
          (dk, "dk", "kv"), (dv, "dv", "kv"), (ws, "ws", "ws"))
    _call("lh_attention_bwd_indexed", ctypes.byref(pr), _p(q), _p(k), _p(v), _p(qpyr), _p(kpyr), _p(vpyr),
          _p(idx), _p(slot), _p(os_), _p(lse), _p(dout), _p(dq), _p(dk), _p(dv), _p(ws),
          _nbytes(ws) if ws_bytes is None else ws_bytes, _stream(stream))


# ---------------------------------------------------------------- allocation helpers

def selection_heads(pr) -> int:
    """Heads of idx, slot, ks, vs (and dks, dvs): Hkv with LH_FLAG_GQA_SHARED, else Hq."""
    return pr.Hkv if pr.flags & LH_FLAG_GQA_SHARED else pr.Hq


def workspace(pr, op, device="cuda"):
    """A device byte buffer of lh_workspace_bytes(pr, op) bytes (None if zero)."""
    n = lh_workspace_bytes(pr, op)
    return torch.empty(max(n, 1), dtype=torch.uint8, device=device)


def attention_forward(q, k, v, p, L, k_budget, scale=0.0, flags=0, stream=None):
    """Allocates the outputs and runs lh_attention_fwd. q [B,N,Hq,D], k/v [B,N,Hkv,D] on the
    device. Returns (pr, dict of o and the forward state)."""
    B, N, Hq, D = q.shape
    Hkv = k.shape[2]
    pr = problem(B, N, Hq, Hkv, D, p, L, k_budget, q.dtype, scale, flags)
    st = lh_check(pr)
    if st != LH_OK:
        raise LighthouseError(f"lh_check: {lh_status_str(st)}: {lh_last_error()}")
    S, Ptot = lh_subseq_len(pr), lh_pyramid_rows(pr)
    Hs = selection_heads(pr)
    dev = q.device
    out = dict(
        o=torch.empty_like(q),
        idx=torch.empty(B, Hs, S, dtype=torch.int32, device=dev),
        slot=torch.empty(B, Hs, Ptot, dtype=torch.int32, device=dev),
        qs=torch.empty(B, Hq, S, D, dtype=q.dtype, device=dev),
        ks=torch.empty(B, Hs, S, D, dtype=q.dtype, device=dev),
        vs=torch.empty(B, Hs, S, D, dtype=q.dtype, device=dev),
        os=torch.empty(B, Hq, S, D, dtype=q.dtype, device=dev),
        lse=torch.empty(B, Hq, S, dtype=torch.float32, device=dev),
    )
    ws = workspace(pr, LH_OP_ATTENTION_FWD, dev)
    lh_attention_fwd(pr, q, k, v, out["o"], out["idx"], out["slot"], out["qs"], out["ks"], out["vs"], out["os"],
                     out["lse"], ws, stream=stream)
    out["ws"] = ws
    return pr, out


def attention_forward_indexed(q, k, v, p, L, k_budget, scale=0.0, flags=0, stream=None):
    """As attention_forward, through lh_attention_fwd_indexed: the state keeps the pyramid
    (qpyr, kpyr, vpyr) instead of the gathered rows."""
    B, N, Hq, D = q.shape
    Hkv = k.shape[2]
    pr = problem(B, N, Hq, Hkv, D, p, L, k_budget, q.dtype, scale, flags)
    st = lh_check(pr)
    if st != LH_OK:
        raise LighthouseError(f"lh_check: {lh_status_str(st)}: {lh_last_error()}")
    S, Ptot = lh_subseq_len(pr), lh_pyramid_rows(pr)
    Hs = selection_heads(pr)
    R = max(Ptot - N, 1)
    dev = q.device
    out = dict(
        o=torch.empty_like(q),
        idx=torch.empty(B, Hs, S, dtype=torch.int32, device=dev),
        slot=torch.empty(B, Hs, Ptot, dtype=torch.int32, device=dev),
        qpyr=torch.empty(B, R, Hq, D, dtype=q.dtype, device=dev),
        kpyr=torch.empty(B, R, Hkv, D, dtype=q.dtype, device=dev),
        vpyr=torch.empty(B, R, Hkv, D, dtype=q.dtype, device=dev),
        os=torch.empty(B, Hq, S, D, dtype=q.dtype, device=dev),
        lse=torch.empty(B, Hq, S, dtype=torch.float32, device=dev),
    )
    ws = workspace(pr, LH_OP_ATTENTION_FWD_INDEXED, dev)
    lh_attention_fwd_indexed(pr, q, k, v, out["o"], out["idx"], out["slot"], out["qpyr"], out["kpyr"],
                             out["vpyr"], out["os"], out["lse"], ws, stream=stream)
    out["ws"] = ws
    return pr, out


def attention_backward_indexed(pr, q, k, v, state, dout, stream=None):
    """Allocates dq, dk, dv and runs lh_attention_bwd_indexed from attention_forward_indexed."""
    B, N, Hq, D = dout.shape
    dq = torch.empty_like(dout)
    dk = torch.empty(B, N, pr.Hkv, D, dtype=dout.dtype, device=dout.device)
    dv = torch.empty_like(dk)
    ws = workspace(pr, LH_OP_ATTENTION_BWD, dout.device)
    lh_attention_bwd_indexed(pr, q, k, v, state["qpyr"], state["kpyr"], state["vpyr"], state["idx"],
                             state["slot"], state["os"], state["lse"], dout, dq, dk, dv, ws, stream=stream)
    return dq, dk, dv


def attention_backward(pr, state, dout, stream=None):
    """Allocates dq, dk, dv and runs lh_attention_bwd from the state of attention_forward."""
    B, N, Hq, D = dout.shape
    dq = torch.empty_like(dout)
    dk = torch.empty(B, N, pr.Hkv, D, dtype=dout.dtype, device=dout.device)
    dv = torch.empty_like(dk)
    ws = workspace(pr, LH_OP_ATTENTION_BWD, dout.device)
    lh_attention_bwd(pr, state["idx"], state["slot"], state["qs"], state["ks"], state["vs"], state["os"],
                     state["lse"], dout, dq, dk, dv, ws, stream=stream)
    return dq, dk, dv
