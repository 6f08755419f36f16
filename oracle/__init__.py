"""CPU oracle of the Lighthouse attention hot path (arXiv 2605.06554).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's CPU-baseline leg use
this package to check and time the GPU path; the product path never imports it. It shares no
code with the HIP library. The arithmetic lives in ``lh_oracle.c`` (fp64, OpenMP over rows);
this module only marshals numpy arrays to it.

Arrays are float64 numpy arrays holding exact images of the stored inputs (bf16 or fp32):
q ``[B, N, Hq, D]``, k and v ``[B, N, Hkv, D]``. Query head ``hq`` uses KV head
``hq // (Hq // Hkv)``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "lh_oracle.c")
_LIB = os.path.join(_HERE, "liblh_oracle.so")

F32, BF16, F64 = 0, 1, 2  # F64: unrounded pooled storage (finite-difference pins)
REPLACE_PARENTS = 1
STRATIFIED = 2
STRAT_CHUNK = 2048  # chunk of the stratified selection (App. D.2)
# One selection per KV group (GQA-shared): the group's query score stream is the elementwise max
# of its query heads' streams, combined with the KV head's stream by the same max as Eq. topk
# combines s_QK and s_KQ. A layer-level flag: the per-head functions above do not see it.
GQA_SHARED = 4


def build(force: bool = True) -> str:
    """Compiles lh_oracle.c into liblh_oracle.so with gcc (plain -O2, OpenMP)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-std=c11", "-O2", "-fopenmp", "-fPIC", "-shared",
                               "-Wall", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


class _Head(ctypes.Structure):
    _fields_ = [("N", ctypes.c_int64), ("D", ctypes.c_int32), ("p", ctypes.c_int32),
                ("L", ctypes.c_int32), ("k", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("flags", ctypes.c_uint32)]


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB):
        build(force=True)
    lib = ctypes.CDLL(_LIB)
    P = ctypes.c_void_p
    i64, i32, dbl = ctypes.c_int64, ctypes.c_int32, ctypes.c_double
    H = ctypes.POINTER(_Head)
    sig = {
        "lho_check": (ctypes.c_int, [H]),
        "lho_level_rows": (i64, [H, ctypes.c_int]),
        "lho_level_offset": (i64, [H, ctypes.c_int]),
        "lho_pyramid_rows": (i64, [H]),
        "lho_round_bf16": (dbl, [dbl]),
        "lho_pool": (None, [H, P, i64, P]),
        "lho_scores": (None, [H, P, i64, P]),
        "lho_select": (i64, [H, P, P, P, i64, P]),
        "lho_gather": (None, [H, P, P, i64, P]),
        "lho_sdpa_fwd": (None, [i64, ctypes.c_int, dbl, P, P, P, P, P, i64, i64]),
        "lho_sdpa_fwd_rows": (None, [i64, ctypes.c_int, dbl, P, P, P, P, P, P, i64]),
        "lho_sdpa_bwd_dq_rows": (None, [i64, ctypes.c_int, dbl, P, P, P, P, P, P, P, P, i64]),
        "lho_sdpa_bwd": (None, [i64, ctypes.c_int, dbl, P, P, P, P, P, P, P, P, P,
                                i64, i64, i64, i64]),
        "lho_scatter": (None, [H, P, i64, P, P, i64]),
        "lho_scatter_bwd": (None, [H, P, i64, P, i64, P]),
        "lho_gather_pool_bwd": (None, [H, P, i64, P, P, i64]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


@dataclass(frozen=True)
class Head:
    """One (batch, query head) problem: base length N, head dim D, pooling factor p,
    L levels, k parents per level, storage dtype of pooled entries, flags."""
    N: int
    D: int
    p: int
    L: int
    k: int
    dtype: int = BF16
    flags: int = 0

    def c(self) -> _Head:
        return _Head(self.N, self.D, self.p, self.L, self.k, self.dtype, self.flags)

    def check(self) -> int:
        return _load().lho_check(ctypes.byref(self.c()))

    def level_rows(self, l: int) -> int:
        return _load().lho_level_rows(ctypes.byref(self.c()), l)

    def level_offset(self, l: int) -> int:
        return _load().lho_level_offset(ctypes.byref(self.c()), l)

    @property
    def ptot(self) -> int:
        return _load().lho_pyramid_rows(ctypes.byref(self.c()))


def round_bf16(x: float) -> float:
    return _load().lho_round_bf16(float(x))


def _rows(x: np.ndarray):
    """(pointer, row stride) of a 2-D float64 view whose rows are contiguous."""
    assert x.dtype == np.float64 and x.ndim == 2 and x.strides[1] == 8
    return x.ctypes.data, x.strides[0] // 8


def pool(h: Head, x: np.ndarray) -> np.ndarray:
    """Pyramid [Ptot, D] of one head slice x [N, D] (Eq. pool)."""
    out = np.empty((h.ptot, h.D), np.float64)
    p, ld = _rows(x)
    _load().lho_pool(ctypes.byref(h.c()), p, ld, _ptr(out))
    return out


def scores(h: Head, x: np.ndarray) -> np.ndarray:
    """fp32 scores [Ptot] of one head slice x [N, D] (Eqs. score-base, score-pool)."""
    out = np.empty(h.ptot, np.float32)
    p, ld = _rows(x)
    _load().lho_scores(ctypes.byref(h.c()), p, ld, _ptr(out))
    return out


def select(h: Head, s_qk: np.ndarray, s_kq: np.ndarray):
    """(idx [S] int32 in causal order, slot [Ptot] int32) from the two fp32 score streams."""
    s_qk = np.ascontiguousarray(s_qk, np.float32)
    s_kq = np.ascontiguousarray(s_kq, np.float32)
    cap = h.ptot
    idx = np.empty(cap, np.int32)
    slot = np.empty(cap, np.int32)
    S = _load().lho_select(ctypes.byref(h.c()), _ptr(s_qk), _ptr(s_kq), _ptr(idx), cap, _ptr(slot))
    if S < 0:
        raise RuntimeError("lho_select failed")
    return idx[:S].copy(), slot


def gather(h: Head, pyr: np.ndarray, idx: np.ndarray) -> np.ndarray:
    idx = np.ascontiguousarray(idx, np.int32)
    out = np.empty((len(idx), h.D), np.float64)
    _load().lho_gather(ctypes.byref(h.c()), _ptr(np.ascontiguousarray(pyr)), _ptr(idx), len(idx), _ptr(out))
    return out


def sdpa_fwd(qs, ks, vs, scale: float, rows=None, row_list=None):
    """Causal SDPA over the gathered order (Eqs. sdpa, attn-sub). Returns (os, lse); only rows
    in ``rows = (r0, r1)`` and, if given, the rows listed in ``row_list`` are computed (others
    are left 0). With only ``row_list`` given, only those rows are computed."""
    qs, ks, vs = (np.ascontiguousarray(a, np.float64) for a in (qs, ks, vs))
    S, D = qs.shape
    os_ = np.zeros((S, D), np.float64)
    lse = np.zeros(S, np.float64)
    if rows is not None or row_list is None:
        r0, r1 = rows if rows is not None else (0, S)
        _load().lho_sdpa_fwd(S, D, scale, _ptr(qs), _ptr(ks), _ptr(vs), _ptr(os_), _ptr(lse), r0, r1)
    if row_list is not None:
        rl = np.ascontiguousarray(row_list, np.int64)
        assert rl.size == 0 or (rl.min() >= 0 and rl.max() < S)
        _load().lho_sdpa_fwd_rows(S, D, scale, _ptr(qs), _ptr(ks), _ptr(vs), _ptr(os_), _ptr(lse),
                                  _ptr(rl), rl.size)
    return os_, lse


def sdpa_bwd(qs, ks, vs, os_, lse, dos, scale: float, qrows=None, krows=None):
    """Adjoint of sdpa_fwd: (dqs, dks, dvs) for rows qrows=(q0,q1) of dqs and krows=(k0,k1) of
    dks, dvs. os_ and lse must be exact for every row the requested outputs depend on."""
    qs, ks, vs, os_, dos = (np.ascontiguousarray(a, np.float64) for a in (qs, ks, vs, os_, dos))
    lse = np.ascontiguousarray(lse, np.float64)
    S, D = qs.shape
    q0, q1 = qrows if qrows is not None else (0, S)
    k0, k1 = krows if krows is not None else (0, S)
    dqs, dks, dvs = (np.zeros((S, D), np.float64) for _ in range(3))
    _load().lho_sdpa_bwd(S, D, scale, _ptr(qs), _ptr(ks), _ptr(vs), _ptr(os_), _ptr(lse), _ptr(dos),
                         _ptr(dqs), _ptr(dks), _ptr(dvs), q0, q1, k0, k1)
    return dqs, dks, dvs


def sdpa_bwd_dq_rows(qs, ks, vs, os_, lse, dos, scale: float, row_list, dqs=None):
    """dq of sdpa_bwd for the listed rows only (os_ and lse exact for those rows), written
    into dqs (a new zero array if None)."""
    qs, ks, vs, os_, dos = (np.ascontiguousarray(a, np.float64) for a in (qs, ks, vs, os_, dos))
    lse = np.ascontiguousarray(lse, np.float64)
    S, D = qs.shape
    if dqs is None:
        dqs = np.zeros((S, D), np.float64)
    assert dqs.shape == (S, D) and dqs.dtype == np.float64 and dqs.flags.c_contiguous
    rl = np.ascontiguousarray(row_list, np.int64)
    assert rl.size == 0 or (rl.min() >= 0 and rl.max() < S)
    _load().lho_sdpa_bwd_dq_rows(S, D, scale, _ptr(qs), _ptr(ks), _ptr(vs), _ptr(os_), _ptr(lse), _ptr(dos),
                                 _ptr(dqs), _ptr(rl), rl.size)
    return dqs


def scatter(h: Head, idx, os_) -> np.ndarray:
    """O [N, D] (Eqs. fanout, scatter)."""
    idx = np.ascontiguousarray(idx, np.int32)
    os_ = np.ascontiguousarray(os_, np.float64)
    out = np.empty((h.N, h.D), np.float64)
    _load().lho_scatter(ctypes.byref(h.c()), _ptr(idx), len(idx), _ptr(os_), _ptr(out), h.D)
    return out


def scatter_bwd(h: Head, idx, dout: np.ndarray) -> np.ndarray:
    idx = np.ascontiguousarray(idx, np.int32)
    out = np.empty((len(idx), h.D), np.float64)
    p, ld = _rows(dout)
    _load().lho_scatter_bwd(ctypes.byref(h.c()), _ptr(idx), len(idx), p, ld, _ptr(out))
    return out


def gather_pool_bwd(h: Head, idx, dxs: np.ndarray, dx: np.ndarray | None = None) -> np.ndarray:
    """Adds the gather+pool adjoint of dxs [S, D] into dx [N, D] (new zero array if None)."""
    idx = np.ascontiguousarray(idx, np.int32)
    dxs = np.ascontiguousarray(dxs, np.float64)
    if dx is None:
        dx = np.zeros((h.N, h.D), np.float64)
    p, ld = _rows(dx)
    _load().lho_gather_pool_bwd(ctypes.byref(h.c()), _ptr(idx), len(idx), _ptr(dxs), p, ld)
    return dx


# ------------------------------------------------------------------ whole layer (small sizes)

def default_scale(D: int, scale: float = 0.0) -> float:
    return scale if scale != 0.0 else 1.0 / np.sqrt(D)


def head_forward(h: Head, scale: float, q: np.ndarray, k: np.ndarray, v: np.ndarray):
    """One (b, hq) problem end to end. q, k, v: [N, D] float64 head slices."""
    s_qk = scores(h, q)
    s_kq = scores(h, k)
    idx, slot = select(h, s_qk, s_kq)
    qs = gather(h, pool(h, q), idx)
    ks = gather(h, pool(h, k), idx)
    vs = gather(h, pool(h, v), idx)
    os_, lse = sdpa_fwd(qs, ks, vs, scale)
    o = scatter(h, idx, os_)
    return dict(s_qk=s_qk, s_kq=s_kq, idx=idx, slot=slot, qs=qs, ks=ks, vs=vs, os=os_, lse=lse, o=o)


def group_forward(h: Head, scale: float, qg: list, k: np.ndarray, v: np.ndarray):
    """One (b, KV group) problem with a shared selection. qg: the group's query-head slices
    [N, D]; k, v: the KV head's slices. The selection ranks by max(max over the group of
    s_QK, s_KQ); every query head attends over the group's gathered K~, V~."""
    s_qk_heads = [scores(h, q) for q in qg]
    s_qk = np.maximum.reduce(s_qk_heads)
    s_kq = scores(h, k)
    idx, slot = select(h, s_qk, s_kq)
    ks = gather(h, pool(h, k), idx)
    vs = gather(h, pool(h, v), idx)
    heads = []
    for q, sq in zip(qg, s_qk_heads):
        qs = gather(h, pool(h, q), idx)
        os_, lse = sdpa_fwd(qs, ks, vs, scale)
        heads.append(dict(s_qk=sq, qs=qs, os=os_, lse=lse, o=scatter(h, idx, os_)))
    return dict(idx=idx, slot=slot, s_kq=s_kq, ks=ks, vs=vs, heads=heads)


def layer_forward(q, k, v, p, L, kk, dtype=BF16, scale=0.0, flags=0):
    """Whole layer for small problems: q [B,N,Hq,D], k/v [B,N,Hkv,D] float64.
    Returns a dict of per-(b,hq) results stacked as [B, Hq, ...] plus o [B,N,Hq,D]. With
    GQA_SHARED in flags, idx, slot, ks and vs are per KV head: [B, Hkv, ...]."""
    B, N, Hq, D = q.shape
    Hkv = k.shape[2]
    G = Hq // Hkv
    if flags & GQA_SHARED:
        return _layer_forward_shared(q, k, v, p, L, kk, dtype, scale, flags & ~GQA_SHARED)
    h = Head(N, D, p, L, kk, dtype, flags)
    sc = default_scale(D, scale)
    res = [[head_forward(h, sc, q[b, :, hq, :], k[b, :, hq // G, :], v[b, :, hq // G, :])
            for hq in range(Hq)] for b in range(B)]
    out = {key: np.stack([np.stack([res[b][hq][key] for hq in range(Hq)]) for b in range(B)])
           for key in ("s_qk", "idx", "slot", "qs", "ks", "vs", "os", "lse")}
    out["s_kq"] = np.stack([np.stack([res[b][g * G]["s_kq"] for g in range(Hkv)]) for b in range(B)])
    out["o"] = np.stack([np.stack([res[b][hq]["o"] for hq in range(Hq)], axis=1) for b in range(B)])
    out["head"] = h
    out["scale"] = sc
    return out


def _layer_forward_shared(q, k, v, p, L, kk, dtype, scale, flags):
    B, N, Hq, D = q.shape
    Hkv = k.shape[2]
    G = Hq // Hkv
    h = Head(N, D, p, L, kk, dtype, flags)
    sc = default_scale(D, scale)
    res = [[group_forward(h, sc, [q[b, :, g * G + t, :] for t in range(G)], k[b, :, g, :], v[b, :, g, :])
            for g in range(Hkv)] for b in range(B)]
    out = {key: np.stack([np.stack([res[b][g][key] for g in range(Hkv)]) for b in range(B)])
           for key in ("idx", "slot", "s_kq", "ks", "vs")}
    for key in ("s_qk", "qs", "os", "lse"):
        out[key] = np.stack([np.stack([res[b][hq // G]["heads"][hq % G][key] for hq in range(Hq)])
                             for b in range(B)])
    out["o"] = np.stack([np.stack([res[b][hq // G]["heads"][hq % G]["o"] for hq in range(Hq)], axis=1)
                         for b in range(B)])
    out["head"] = h
    out["scale"] = sc
    out["shared"] = True
    return out


def layer_backward(fwd, dout):
    """Backward of layer_forward from dout [B,N,Hq,D] float64: (dq, dk, dv, dos, dqs, dks, dvs).
    With a shared selection, dks and dvs are per KV head: the sums over the group's query heads
    of each head's gradient of the shared K~, V~."""
    if fwd.get("shared"):
        return _layer_backward_shared(fwd, dout)
    h = fwd["head"]
    sc = fwd["scale"]
    B, Hq, S = fwd["idx"].shape
    N, D = h.N, h.D
    Hkv = fwd["s_kq"].shape[1]
    G = Hq // Hkv
    dq = np.zeros((B, N, Hq, D))
    dk = np.zeros((B, N, Hkv, D))
    dv = np.zeros((B, N, Hkv, D))
    dos = np.zeros((B, Hq, S, D))
    dqs = np.zeros((B, Hq, S, D))
    dks = np.zeros((B, Hq, S, D))
    dvs = np.zeros((B, Hq, S, D))
    for b in range(B):
        for hq in range(Hq):
            idx = fwd["idx"][b, hq]
            dos[b, hq] = scatter_bwd(h, idx, np.ascontiguousarray(dout[b, :, hq, :]))
            dqs[b, hq], dks[b, hq], dvs[b, hq] = sdpa_bwd(
                fwd["qs"][b, hq], fwd["ks"][b, hq], fwd["vs"][b, hq], fwd["os"][b, hq],
                fwd["lse"][b, hq], dos[b, hq], sc)
            tq = np.zeros((N, D))
            gather_pool_bwd(h, idx, dqs[b, hq], tq)
            dq[b, :, hq, :] = tq
            tk = np.zeros((N, D))
            gather_pool_bwd(h, idx, dks[b, hq], tk)
            dk[b, :, hq // G, :] += tk
            tv = np.zeros((N, D))
            gather_pool_bwd(h, idx, dvs[b, hq], tv)
            dv[b, :, hq // G, :] += tv
    return dict(dq=dq, dk=dk, dv=dv, dos=dos, dqs=dqs, dks=dks, dvs=dvs)


def _layer_backward_shared(fwd, dout):
    h = fwd["head"]
    sc = fwd["scale"]
    B, Hq, S = fwd["qs"].shape[:3]
    Hkv = fwd["idx"].shape[1]
    G = Hq // Hkv
    N, D = h.N, h.D
    dq = np.zeros((B, N, Hq, D))
    dk = np.zeros((B, N, Hkv, D))
    dv = np.zeros((B, N, Hkv, D))
    dos = np.zeros((B, Hq, S, D))
    dqs = np.zeros((B, Hq, S, D))
    dks = np.zeros((B, Hkv, S, D))
    dvs = np.zeros((B, Hkv, S, D))
    for b in range(B):
        for g in range(Hkv):
            idx = fwd["idx"][b, g]
            for hq in range(g * G, (g + 1) * G):
                dos[b, hq] = scatter_bwd(h, idx, np.ascontiguousarray(dout[b, :, hq, :]))
                dqs[b, hq], tk, tv = sdpa_bwd(fwd["qs"][b, hq], fwd["ks"][b, g], fwd["vs"][b, g],
                                              fwd["os"][b, hq], fwd["lse"][b, hq], dos[b, hq], sc)
                dks[b, g] += tk
                dvs[b, g] += tv
                tq = np.zeros((N, D))
                gather_pool_bwd(h, idx, dqs[b, hq], tq)
                dq[b, :, hq, :] = tq
            tk = np.zeros((N, D))
            gather_pool_bwd(h, idx, dks[b, g], tk)
            dk[b, :, g, :] = tk
            tv = np.zeros((N, D))
            gather_pool_bwd(h, idx, dvs[b, g], tv)
            dv[b, :, g, :] = tv
    return dict(dq=dq, dk=dk, dv=dv, dos=dos, dqs=dqs, dks=dks, dvs=dvs)
