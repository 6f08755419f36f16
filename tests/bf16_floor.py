"""Error floor of bf16 arithmetic on the attention path (test infrastructure).

A bf16 layer stores every Q/K/V-like tensor and gradient of the interface in bf16, and a bf16
matrix-core SDPA multiplies bf16 operands. Even an implementation that is exact apart from those
roundings differs from the fp64 oracle, by an amount that grows with the magnitude of what is
rounded: a gradient of a coarse pyramid entry sums up to p^(L-1) rows of dO (Sec. 3.6, the
adjoint of Eq. scatter), so it reaches tens, where one bf16 rounding moves a value by up to
0.125.

This module recomputes a head's layer from the oracle's own gathered rows (which the GPU path
reproduces bit for bit) with exactly these roundings to bf16 and fp64 everywhere else:
  forward:  the softmax weights before their product with V~; O~; O;
  backward: dO~; the softmax weights before P^T dO~; dS before dS K~ and dS^T Q~; dQ~, dK~,
            dV~; dQ, dK, dV.
Its distance to the oracle is the floor: what a correct bf16 implementation of the stated
design cannot avoid. The parity tests report it beside each tensor's raw error and accept a
bf16 tensor that misses the raw bar only if its error stays within a small multiple of this
floor (see ``parity.py``).

The products run on torch's CPU float64 kernels in row blocks, so the full c4 sequence
(S = 54,272) fits in a few GB of host memory. Nothing here is shared with the HIP library.
"""
from __future__ import annotations

import numpy as np
import torch

import oracle

BLOCK = 1024


def bf16(x: torch.Tensor) -> torch.Tensor:
    """Round float64 values to bf16 (nearest, ties to even) and back. torch converts through
    fp32, so a value within 2^-24 relative of a bf16 tie can round the other way: immaterial
    for an error floor."""
    return x.to(torch.bfloat16).to(torch.float64)


def _t(a) -> torch.Tensor:
    return torch.as_tensor(np.ascontiguousarray(a, np.float64))


def _blocks(rows):
    """Consecutive chunks of at most BLOCK entries of a sorted row list."""
    for i in range(0, len(rows), BLOCK):
        yield rows[i:i + BLOCK]


def sdpa_fwd(qs, ks, vs, scale: float, rows=None):
    """(os, lse) of causal SDPA with the softmax weights rounded before P V and O~ rounded, for
    the sorted query rows `rows` (all rows by default; other rows are left 0)."""
    q, k, v = _t(qs), _t(ks), _t(vs)
    S = q.shape[0]
    rows = np.arange(S) if rows is None else np.asarray(rows, np.int64)
    os_ = torch.zeros_like(q)
    lse = torch.zeros(S, dtype=torch.float64)
    for ch in _blocks(rows):
        r1 = int(ch[-1]) + 1
        rt = torch.as_tensor(ch)
        a = (q[rt] @ k[:r1].T) * scale
        a.masked_fill_(torch.arange(r1)[None, :] > rt[:, None], float("-inf"))
        mu = a.max(dim=1, keepdim=True).values
        z = torch.exp(a - mu).sum(dim=1, keepdim=True)
        lse[rt] = (mu + torch.log(z)).squeeze(1)
        # the normalised weights are rounded: a weight of exactly 1 (the row maximum relative
        # to itself) would hide the rounding of a row's dominant weight, which no running-max
        # implementation avoids
        os_[rt] = bf16(bf16(torch.exp(a - lse[rt, None])) @ v[:r1])
    return os_.numpy(), lse.numpy()


def sdpa_bwd(qs, ks, vs, os_b, lse, dos_b, scale: float, qrows=None, krange=None):
    """(dqs rounded to bf16, dks and dvs unrounded) from bf16 os and dos, with P and dS rounded
    before their products. dks and dvs are left unrounded because a selection head shared by
    several query heads sums their gradients before its one rounding. dqs is computed for the
    sorted query rows `qrows` and dks, dvs for the key rows [k0, k1) = `krange` (all rows by
    default); os_b, lse and dos_b must hold every row these depend on."""
    q, k, v = _t(qs), _t(ks), _t(vs)
    o, do = _t(os_b), _t(dos_b)
    lse = torch.as_tensor(np.asarray(lse, np.float64))
    S = q.shape[0]
    delta = (do * o).sum(dim=1)
    dq = torch.zeros_like(q)
    dk = torch.zeros_like(q)
    dv = torch.zeros_like(q)
    full = qrows is None and krange is None
    qrows = np.arange(S) if qrows is None else np.asarray(qrows, np.int64)
    k0, k1 = (0, S) if krange is None else krange

    def tile(rt, c0, c1):
        a = (q[rt] @ k[c0:c1].T) * scale
        p = torch.exp(a - lse[rt, None])
        p.masked_fill_(torch.arange(c0, c1)[None, :] > rt[:, None], 0.0)
        dp = do[rt] @ v[c0:c1].T
        return p, bf16(p * (dp - delta[rt, None]))

    for ch in _blocks(qrows):
        rt = torch.as_tensor(ch)
        r1 = int(ch[-1]) + 1
        p, ds = tile(rt, 0, r1)
        dq[rt] = (ds @ k[:r1]) * scale
        if full:
            dk[:r1] += ds.T @ q[rt]
            dv[:r1] += bf16(p).T @ do[rt]
    if not full and k1 > k0:
        for ch in _blocks(np.arange(k0, S)):
            rt = torch.as_tensor(ch)
            c1 = min(k1, int(ch[-1]) + 1)
            p, ds = tile(rt, k0, c1)
            dk[k0:c1] += ds.T @ q[rt]
            dv[k0:c1] += bf16(p).T @ do[rt]
    return bf16(dq).numpy(), (dk * scale).numpy(), dv.numpy()


def round_bf16(a) -> np.ndarray:
    return bf16(_t(a)).numpy()


def layer(f: dict, dout: np.ndarray, backward: bool = True) -> dict:
    """The floor emulation of a whole layer from the oracle's forward dict ``f`` (of
    ``oracle.layer_forward``; its gathered rows are exact) and dout [B, N, Hq, D]. Returns the
    tensors of the oracle's layout: os, lse, o and, with ``backward``, dos, dqs, dks, dvs, dq,
    dk, dv. The selection head of query head hq is hq // (Hq / Hs); with one selection per KV
    group the group's dK~, dV~ sum its query heads before their rounding, and every KV head sums
    its selection heads' pooled gradients in fp64 before the final rounding, as the layer's
    one-rounding adjoints do."""
    h, sc = f["head"], f["scale"]
    B, Hq, S, D = f["qs"].shape
    Hs = f["idx"].shape[1]
    Hkv = f["s_kq"].shape[1]
    N = h.N
    Gs, G = Hq // Hs, Hq // Hkv
    out = dict(os=np.zeros((B, Hq, S, D)), lse=np.zeros((B, Hq, S)), o=np.zeros((B, N, Hq, D)))
    if backward:
        out.update(dos=np.zeros((B, Hq, S, D)), dqs=np.zeros((B, Hq, S, D)), dks=np.zeros((B, Hs, S, D)),
                   dvs=np.zeros((B, Hs, S, D)), dq=np.zeros((B, N, Hq, D)))
        dk, dv = np.zeros((B, N, Hkv, D)), np.zeros((B, N, Hkv, D))
    for b in range(B):
        for hs in range(Hs):
            idx = f["idx"][b, hs]
            dks_u, dvs_u = np.zeros((S, D)), np.zeros((S, D))
            for hq in range(hs * Gs, (hs + 1) * Gs):
                out["os"][b, hq], out["lse"][b, hq] = sdpa_fwd(f["qs"][b, hq], f["ks"][b, hs], f["vs"][b, hs], sc)
                out["o"][b, :, hq] = round_bf16(oracle.scatter(h, idx, out["os"][b, hq]))
                if not backward:
                    continue
                dos_b = round_bf16(oracle.scatter_bwd(h, idx, np.ascontiguousarray(dout[b, :, hq], np.float64)))
                out["dos"][b, hq] = dos_b
                dqs, tk, tv = sdpa_bwd(f["qs"][b, hq], f["ks"][b, hs], f["vs"][b, hs], out["os"][b, hq],
                                       out["lse"][b, hq], dos_b, sc)
                out["dqs"][b, hq] = dqs
                out["dq"][b, :, hq] = round_bf16(oracle.gather_pool_bwd(h, idx, dqs))
                dks_u += tk
                dvs_u += tv
            if backward:
                out["dks"][b, hs] = round_bf16(dks_u)
                out["dvs"][b, hs] = round_bf16(dvs_u)
                g = hs * Gs // G
                oracle.gather_pool_bwd(h, idx, out["dks"][b, hs], dk[b, :, g])
                oracle.gather_pool_bwd(h, idx, out["dvs"][b, hs], dv[b, :, g])
    if backward:
        out["dk"] = round_bf16(dk)
        out["dv"] = round_bf16(dv)
    return out
