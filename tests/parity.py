"""Comparison helpers for the GPU parity tests.

Indices, slots, fp32 scores, pooled rows and gathered rows are compared bit for bit.

Floating-point outputs are held to the stated bar first: raw max-abs |gpu - ref| <= 1e-4 for the
fp32 path (and for the fp32 log-sum-exp of either path), <= 2e-2 for bf16 tensors.

A bf16 tensor cannot always meet 2e-2: storing a value of magnitude 8 or more in bf16 moves it by
up to 2^-5 (half a unit in the last place), and the gradients of coarse pyramid entries, which sum
up to p^(L-1) rows of dO, reach tens. Such a tensor passes only against its bf16 floor, the error
that bf16 rounding alone produces, reported beside the raw error (``bf16_floor.py``):
  * a stage that sums exact bf16 inputs in fp32 and rounds once (scatter, its adjoint, the
    gather and pool adjoint) has the floor of rounding the exact result, element by element:
    every element must satisfy |gpu - ref| <= 2 * |bf16(ref) - ref| (or the raw bar);
  * the attention and the whole layer have the floor of an emulation that performs exactly the
    design's roundings (stored tensors, and the softmax weights and dS before their products) in
    otherwise exact arithmetic: per head slice, max |gpu - ref| <= 2 * floor, where floor is
    the larger of max |emulated - ref| and half a bf16 ulp of the slice's largest |ref|.
A wrong mask, index, scale or dropped term gives errors the size of the values themselves, tens
to hundreds of times these floors. No fp32 tensor is given a floor.

Every comparison is recorded (raw max-abs, magnitude, floor, basis) and printed in the pytest
terminal summary; with LH_PARITY_JSON set, the records are also written to that file.
"""
from __future__ import annotations

import numpy as np
import torch

import bf16_floor
import oracle

TOL = {"fp32": 1e-4, "bf16": 2e-2}
FLOOR_MULT = 2.0
RECORDS: list = []
CURRENT = {"test": ""}


def to64(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu", torch.float64).numpy()


def _np(x) -> np.ndarray:
    return to64(x) if isinstance(x, torch.Tensor) else np.asarray(x, np.float64)


def rounding_floor(ref) -> np.ndarray:
    """Element-wise distance of the exact values to their bf16 rounding (nearest even)."""
    r = np.asarray(ref, np.float64)
    return np.abs(torch.from_numpy(r).to(torch.bfloat16).double().numpy() - r)


def emulated_floor(emu, ref) -> float:
    """The bf16 floor of a tensor from its emulation: the emulation's max-abs distance to the
    oracle, and at least half a bf16 unit in the last place of the tensor's largest value (the
    worst case of storing that value, which one realisation of the roundings can miss)."""
    e = np.asarray(emu, np.float64)
    r = np.asarray(ref, np.float64)
    if not r.size:
        return 0.0
    m = float(np.abs(r).max())
    half_ulp = 2.0 ** (np.floor(np.log2(m)) - 8) if m > 0 else 0.0
    return max(float(np.abs(e - r).max()), half_ulp)


def check_close(name, gpu, ref, dtype, floor=None):
    """Raw max-abs check against TOL[dtype]; a bf16 tensor that misses it is checked against
    FLOOR_MULT times `floor` (a scalar, or an array of the tensor's shape for an element-wise
    floor). Returns the raw max-abs error."""
    g = _np(gpu)
    r = np.asarray(ref, np.float64)
    assert g.shape == r.shape, (name, g.shape, r.shape)
    assert np.isfinite(g).all(), f"{name}: non-finite values"
    tol = TOL[dtype]
    d = np.abs(g - r)
    raw = float(d.max()) if d.size else 0.0
    rec = dict(test=CURRENT["test"], name=name, dtype=dtype, raw=raw,
               max_ref=float(np.abs(r).max()) if r.size else 0.0, floor=None, ratio=None, basis="raw")
    if floor is not None:
        fl = np.broadcast_to(np.asarray(floor, np.float64), d.shape)
        rec["floor"] = float(fl.max()) if fl.size else 0.0
        over = d > tol
        if over.any():  # the ratio that decides: errors past the raw bar over their floor
            with np.errstate(divide="ignore"):
                rec["ratio"] = float((d[over] / fl[over]).max())
    if raw > tol:
        assert dtype == "bf16" and floor is not None, (
            f"{name}: max abs err {raw:.3e} > {tol:g} at {np.unravel_index(int(d.argmax()), d.shape)} "
            f"(|ref| up to {rec['max_ref']:.3e})")
        bound = np.maximum(tol, FLOOR_MULT * fl)
        bad = d > bound
        if bad.any():
            at = np.unravel_index(int(np.argmax(np.where(bad, d / bound, 0.0))), d.shape)
            raise AssertionError(f"{name}: err {d[at]:.3e} > max({tol:g}, {FLOOR_MULT:g} x bf16 floor "
                                 f"{fl[at]:.3e}) at {at} ({int(bad.sum())} of {d.size} elements); "
                                 f"raw max {raw:.3e}")
        rec["basis"] = "floor"
    RECORDS.append(rec)
    return raw


def check_close_heads(name, gpu, ref, dtype, head_axis, emu=None, floor=None):
    """check_close on every slice along `head_axis` (and the batch axis 0). `emu` is a
    floor emulation of the same shape (its per-slice max distance to ref is the slice's floor);
    `floor` an element-wise floor of the same shape."""
    g = _np(gpu)
    r = np.asarray(ref, np.float64)
    worst = 0.0
    for b in range(g.shape[0]):
        for h in range(g.shape[head_axis]):
            gs = np.take(g[b], h, axis=head_axis - 1)
            rs = np.take(r[b], h, axis=head_axis - 1)
            fl = None
            if emu is not None:
                es = np.take(np.asarray(emu, np.float64)[b], h, axis=head_axis - 1)
                fl = emulated_floor(es, rs)
            elif floor is not None:
                fl = np.take(np.asarray(floor, np.float64)[b], h, axis=head_axis - 1)
            worst = max(worst, check_close(f"{name}[{b},{h}]", gs, rs, dtype, fl))
    return worst


def check_equal(name, gpu, ref):
    g = gpu.detach().cpu().numpy() if isinstance(gpu, torch.Tensor) else np.asarray(gpu)
    r = np.asarray(ref)
    assert g.shape == r.shape, (name, g.shape, r.shape)
    if g.dtype == np.float32 or r.dtype == np.float32:
        same = g.astype(np.float32).view(np.uint32) == r.astype(np.float32).view(np.uint32)
    else:
        same = g == r
    assert same.all(), f"{name}: {int((~same).sum())} of {same.size} differ; first at {np.argwhere(~same)[0].tolist()}"


def summary_lines():
    """One line per (test, tensor): the worst raw error over its slices, the floor and ratio at
    that slice, and whether every slice met the raw bar."""
    agg = {}
    for r in RECORDS:
        base = r["name"].split("[")[0]
        key = (r["test"], base)
        a = agg.get(key)
        if a is None:
            agg[key] = a = dict(r, n=0, n_floor=0)
        a["n"] += 1
        a["n_floor"] += r["basis"] == "floor"
        if r["raw"] > a["raw"]:
            a.update(raw=r["raw"], floor=r["floor"], ratio=r["ratio"], max_ref=r["max_ref"])
        if r["ratio"] is not None and (a.get("worst_ratio") is None or r["ratio"] > a["worst_ratio"]):
            a["worst_ratio"] = r["ratio"]
    out = []
    for (test, base), a in agg.items():
        fl = "-" if a["floor"] is None else f"{a['floor']:.2e}"
        wr = "-" if a.get("worst_ratio") is None else f"{a['worst_ratio']:.2f}"
        basis = "raw" if a["n_floor"] == 0 else f"floor in {a['n_floor']}/{a['n']} slices"
        out.append(f"{test.split('::')[-1]:<58} {base:<14} {a['dtype']:<4} raw {a['raw']:.2e} "
                   f"(bar {TOL[a['dtype']]:g}, |ref| {a['max_ref']:.1e}) floor {fl} "
                   f"worst err/floor {wr}  {basis}")
    return out


def check_layer(c, inp, st, grads, f=None, g=None):
    """Every output of the fused layer against the oracle: the selection and gathered rows bit
    for bit (the gathered rows only where the state holds them: the indexed path keeps the
    pyramid instead), the floating-point tensors at the raw bar or, for bf16 tensors that cannot
    meet it, within the bound of their bf16 floor (module docstring)."""
    dq, dk, dv = grads
    q, k, v = (inp[x].double().numpy() for x in ("q", "k", "v"))
    dout = inp["dout"].double().numpy()
    odt = oracle.BF16 if c.dtype == "bf16" else oracle.F32
    if f is None:
        f = oracle.layer_forward(q, k, v, c.p, c.L, c.k, dtype=odt, flags=c.flags)
        g = oracle.layer_backward(f, dout)
    emu = bf16_floor.layer(f, dout) if c.dtype == "bf16" else {}
    check_equal("idx", st["idx"], f["idx"])
    check_equal("slot", st["slot"], f["slot"])
    for key in ("qs", "ks", "vs"):
        if key in st:
            check_equal(key, st[key].double(), f[key])
    check_close_heads("os", st["os"], f["os"], c.dtype, 1, emu=emu.get("os"))
    check_close_heads("lse", st["lse"], f["lse"], "fp32", 1)
    check_close_heads("o", st["o"], f["o"], c.dtype, 2, emu=emu.get("o"))
    check_close_heads("dq", dq, g["dq"], c.dtype, 2, emu=emu.get("dq"))
    check_close_heads("dk", dk, g["dk"], c.dtype, 2, emu=emu.get("dk"))
    check_close_heads("dv", dv, g["dv"], c.dtype, 2, emu=emu.get("dv"))
    return f, g
