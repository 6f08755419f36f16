"""Comparison helpers for the GPU parity tests.

Indices, slots, fp32 scores, pooled rows and gathered rows are compared bit for bit.

Floating-point outputs: the bar is max-abs 1e-4 (fp32 path) or 2e-2 (bf16 path), applied to each
tensor slice after normalising it by its magnitude:
    max |gpu - ref| <= tol * max(1, max |ref|)
For slices whose values stay within [-1, 1] this is exactly the max-abs bar. Larger values
need the normalisation because bf16 keeps 8 significant bits. One rounding of a value in
[32, 64) moves it by up to 0.125. Gradients of coarse pyramid entries are sums of up to
p^(L-1) rows of dO, so they reach such magnitudes. The errors of the gradients of the gathered
queries are set by the largest terms of their sums, not by the element itself. A CPU emulation
of only the standard bf16 roundings of the attention backward reproduces the GPU error on the
spiky test workload: O and dO stored in bf16, and the softmax gradient rounded to bf16 before
its matrix product. So an element-wise relative bar would reject correct bf16 arithmetic. The
normalised bar still catches a wrong mask, index, scale or dropped term, because those errors
have the size of the values themselves.
"""
from __future__ import annotations

import numpy as np
import torch

TOL = {"fp32": 1e-4, "bf16": 2e-2}


def to64(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu", torch.float64).numpy()


def check_close(name, gpu, ref, dtype, report=None):
    """Normalised max-abs check (see the module docstring). Returns (max_abs, normalised)."""
    g = to64(gpu) if isinstance(gpu, torch.Tensor) else np.asarray(gpu, np.float64)
    r = np.asarray(ref, np.float64)
    assert g.shape == r.shape, (name, g.shape, r.shape)
    assert np.isfinite(g).all(), f"{name}: non-finite values"
    tol = TOL[dtype]
    d = np.abs(g - r)
    maxabs = float(d.max()) if d.size else 0.0
    scale = max(1.0, float(np.abs(r).max()) if r.size else 0.0)
    if report is not None:
        report[name] = dict(max_abs=maxabs, max_ref=scale, normalised=maxabs / scale)
    assert maxabs <= tol * scale, (f"{name}: max abs err {maxabs:.3e} > {tol:g} * {scale:.3e} "
                                   f"at {np.unravel_index(int(d.argmax()), d.shape)}")
    return maxabs, maxabs / scale


def check_close_heads(name, gpu, ref, dtype, head_axis, report=None):
    """check_close on every slice along `head_axis` (and the batch axis 0)."""
    g = to64(gpu) if isinstance(gpu, torch.Tensor) else np.asarray(gpu, np.float64)
    r = np.asarray(ref, np.float64)
    worst = 0.0
    for b in range(g.shape[0]):
        for h in range(g.shape[head_axis]):
            gs = np.take(g[b], h, axis=head_axis - 1)
            rs = np.take(r[b], h, axis=head_axis - 1)
            worst = max(worst, check_close(f"{name}[{b},{h}]", gs, rs, dtype, report)[1])
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
