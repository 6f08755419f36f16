"""CPU mirror of the memory kernels' index arithmetic, over their full launch grids.

For every workload shape (the benchmark configs, the shard config and the parity-test configs,
each also with one selection per KV group where a group has several query heads), this test
recomputes each launcher's grid and the per-thread index arithmetic of

    gather_kernel; scatter_long_kernel, scatter_kernel; gather_bwd_long_kernel,
    gather_bwd_group_long_kernel (packed and not), gather_bwd_group_kernel, gather_bwd_kernel;
    scatter_bwd_kernel; pool_score_kernel; the selection workspace of select_kernel and
    order_kernel

from the formulas of their sources, and asserts:
  * every index the kernels use unguarded (slot and idx reads, pyramid and score rows, head
    and column offsets, LDS offsets) lies inside its buffer; reads of gathered rows through a
    slot value are guarded in the kernels by m < S and so only need their head offset checked;
  * every output element is written exactly once (the kernels rely on it: there is no zero
    fill), and the XCD remap of run indices is a bijection;
  * the shape facts (Ptot, S, candidate counts) equal the library's host-side values.
The arrays are built per launch dimension (run index, head-chunk index, batch), which the
address arithmetic combines affinely, so the extremes of each term bound the whole grid.
Any change to the kernels' index math must be mirrored here.
"""
from __future__ import annotations

import numpy as np
import pytest

import workloads

lh = pytest.importorskip("paper_2605_06554_amd")


class Shape:
    """The derived shape of a problem, recomputed from the paper's definitions (Sec. 3.3 level
    sizes, Eq. S-size with the per-level descent)."""

    def __init__(self, c, flags=None):
        self.B, self.N, self.Hq, self.Hkv, self.D = c.B, c.N, c.Hq, c.Hkv, c.D
        self.p, self.L, self.k = (c.p if c.L > 1 else max(c.p, 1)), c.L, c.k
        self.flags = c.flags if flags is None else flags
        self.es = 2 if c.dtype == "bf16" else 4
        self.G = self.Hq // self.Hkv
        shared = bool(self.flags & 4)
        self.Hs = self.Hkv if shared else self.Hq
        self.Gq = self.G if shared else 1
        self.pw = [self.p ** l for l in range(self.L)]
        self.nrow = [self.N // w for w in self.pw]
        self.off = [0]
        for n in self.nrow:
            self.off.append(self.off[-1] + n)
        self.Ptot = self.off[-1]
        self.R = self.Ptot - self.N
        self.P = self.pw[-1]
        cand = [0] * self.L
        npar = [0] * self.L
        cand[self.L - 1] = self.N // self.P
        for l in range(self.L - 1, 0, -1):
            npar[l] = min(cand[l], self.k)
            cand[l - 1] = self.p * npar[l]
        self.cand, self.npar = cand, npar
        self.coff = np.concatenate([[0], np.cumsum(cand)]).tolist()
        self.Scand = self.coff[-1]
        self.S = self.Scand - (sum(npar[1:]) if self.flags & 1 else 0)
        self.CH = 16 // self.es
        self.cs = int(np.log2(self.D // self.CH))
        self.maxsel = max([cand[l] for l in range(1, self.L) if 0 < npar[l] < cand[l]], default=0)

    def problem(self):
        return lh.problem(self.B, self.N, self.Hq, self.Hkv, self.D, self.p, self.L, self.k,
                          lh.LH_BF16 if self.es == 2 else lh.LH_F32, 0.0, self.flags)


def _cases():
    out = []
    allc = {**workloads.CONFIGS, **workloads.SHARD_CONFIGS, **workloads.TEST_CONFIGS}
    for name, c in allc.items():
        out.append((name, c, c.flags))
        if c.Hq > c.Hkv and not c.flags & 4:
            out.append((name + "+shared", c, c.flags | 4))
    return out


CASES = _cases()


def inside(name, lo, hi, size):
    """Every access [lo, hi) (arrays or scalars, in elements) lies in [0, size)."""
    lo, hi = np.min(lo), np.max(hi)
    assert lo >= 0 and hi <= size, f"{name}: accesses [{lo}, {hi}) outside [0, {size})"


def once(name, ids, n):
    """ids (flattened) cover [0, n) exactly once."""
    ids = np.asarray(ids, np.int64).ravel()
    assert ids.size == n and ids.min(initial=0) >= 0 and (n == 0 or ids.max() < n), f"{name}: bad coverage"
    cnt = np.bincount(ids, minlength=n)
    assert (cnt == 1).all(), f"{name}: {int((cnt == 0).sum())} missed, {int((cnt > 1).sum())} repeated"


def xcd(nx):
    """xcd_contiguous(bx, nx) for every bx in [0, nx); nx is a multiple of 8."""
    assert nx % 8 == 0
    bx = np.arange(nx, dtype=np.int64)
    c = (bx & 7) * (nx >> 3) + (bx >> 3)
    once("xcd remap", c, nx)
    return c


@pytest.mark.parametrize("name,c,flags", CASES, ids=[x[0] for x in CASES])
def test_shape_matches_library(name, c, flags):
    s = Shape(c, flags)
    pr = s.problem()
    assert lh.lh_check(pr) == lh.LH_OK, lh.lh_last_error()
    assert lh.lh_pyramid_rows(pr) == s.Ptot
    assert lh.lh_subseq_len(pr) == s.S
    for l in range(s.L):
        assert lh.lh_level_offset(pr, l) == s.off[l]
        assert lh.lh_level_rows(pr, l) == s.nrow[l]


@pytest.mark.parametrize("name,c,flags", CASES, ids=[x[0] for x in CASES])
def test_gather_index_math(name, c, flags):
    s = Shape(c, flags)
    rpb = 256 >> s.cs
    gx = -(-s.S // rpb)
    tid = np.arange(256)
    m = (np.arange(gx)[:, None] * rpb + (tid[None, :] >> s.cs)).ravel()
    cc = np.broadcast_to(tid[None, :] & ((1 << s.cs) - 1), (gx, 256)).ravel()
    live = m < s.S
    m, cc = m[live], cc[live]
    once("gather (m, cc)", m * (1 << s.cs) + cc, s.S << s.cs)
    bh = np.arange(s.B * s.Hq)
    hq, b = bh % s.Hq, bh // s.Hq
    g = hq // s.G
    bs = b * s.Hs + hq // s.Gq
    kv_out = hq % s.Gq == 0
    once("gather K~/V~ writers", bs[kv_out], s.B * s.Hs)
    inside("idx read", bs.min() * s.S, bs.max() * s.S + s.S, s.B * s.Hs * s.S)
    col_hi = cc.max() * s.CH + s.CH
    inside("qs write", 0, (bh.max() * s.S + s.S - 1) * s.D + col_hi, s.B * s.Hq * s.S * s.D)
    inside("ks write", 0, (bs.max() * s.S + s.S - 1) * s.D + col_hi, s.B * s.Hs * s.S * s.D)
    # ids are checked against [0, N + R) before any read
    inside("q read", 0, ((b.max() * s.N + s.N - 1) * s.Hq + hq.max()) * s.D + col_hi, s.B * s.N * s.Hq * s.D)
    inside("k read", 0, ((b.max() * s.N + s.N - 1) * s.Hkv + g.max()) * s.D + col_hi, s.B * s.N * s.Hkv * s.D)
    if s.R:
        inside("qpyr read", 0, ((b.max() * s.R + s.R - 1) * s.Hq + hq.max()) * s.D + col_hi, s.B * s.R * s.Hq * s.D)
        inside("kpyr read", 0, ((b.max() * s.R + s.R - 1) * s.Hkv + g.max()) * s.D + col_hi, s.B * s.R * s.Hkv * s.D)


def _long_tt(s):
    if s.L < 2:
        return 0
    return {4: 2, 2: 3}.get(s.p, 0)


class RunLaunch:
    """run_args + run_grid + the variant choice of launch_scatter_P / launch_gather_bwd_P."""

    def __init__(self, s, scatter, H, Gs, Hsrc, sdiv):
        self.s, self.scatter, self.H, self.Gs, self.Hsrc, self.sdiv = s, scatter, H, Gs, Hsrc, sdiv
        self.run = s.p if s.L > 1 else 1
        self.nruns = s.N // self.run + (1 if scatter else 0)
        self.HC = H << s.cs
        self.bs = min(self.HC, 512)
        self.nx = -(-self.nruns // 8) * 8
        self.gy = -(-self.HC // self.bs)
        self.rpb = 1
        self.vec_slots = s.Ptot % 4 == 0
        tt = _long_tt(s)
        if scatter:
            if tt:
                self.kind, self.RL = "long", (16 if tt == 2 else 8)
                self.nruns = (s.N + self.RL) // self.RL
                self.nx = -(-self.nruns // 8) * 8
            else:
                self.kind, self.RL = "runs", self.run
        else:
            if Gs == 1 and tt:
                self.kind, self.RL = "long", (16 if tt == 2 else 8)
                self.nruns = -(-s.N // self.RL)
                self.nx = -(-self.nruns // 8) * 8
            elif Gs > 1 and s.L > 1 and s.p in (2, 4):
                self.kind, self.RL = "group_long", 8
                self.nruns = -(-s.N // 8)
                self.rpb = 64 // self.HC if self.HC < 64 else 1
                self.nx = -(-(-(-self.nruns // self.rpb)) // 8) * 8
                if self.rpb > 1:
                    self.bs = self.rpb * self.HC
                    self.gy = 1
            else:
                self.kind, self.RL = ("group" if Gs > 1 else "runs"), self.run

    def threads(self):
        """(c, hc) of every live thread."""
        c = xcd(self.nx)
        if self.kind == "group_long" and self.rpb > 1:
            tid = np.arange(self.bs)
            sub = tid // self.HC
            cc = (c[:, None] * self.rpb + sub[None, :]).ravel()
            hc = np.broadcast_to(tid - sub * self.HC, (len(c), self.bs)).ravel()
            live = (cc < self.nruns) & (hc < self.HC)
            return cc[live], hc[live]
        hc = np.arange(self.gy * self.bs)
        return c[c < self.nruns], hc[hc < self.HC]


def _positions(rl, c, r_count, shift):
    """Base positions j = c RL + r - shift of runs c (2-D: [run, r])."""
    return c[:, None] * rl + np.arange(r_count)[None, :] - shift


def _check_run_kernel(s, rl_obj, label):
    """Bounds and coverage of one scatter / gather+pool-adjoint launch."""
    a = rl_obj
    c, hc = a.threads()
    if a.kind == "group_long" and a.rpb > 1:
        pairs = np.stack([c, hc], 1)
        once(f"{label} packed threads", pairs[:, 0] * a.HC + pairs[:, 1], a.nruns * a.HC)
        c = np.unique(c)
        hc = np.arange(a.HC)
    h, cc = hc >> s.cs, hc & ((1 << s.cs) - 1)
    once(f"{label} (h, cc)", hc, a.HC)
    shift = 1 if a.scatter else 0
    RL = a.RL
    j = _positions(RL, c, RL, shift)
    inrange = (j >= 0) & (j < s.N)
    # every output position written exactly once per (h, cc)
    once(f"{label} positions", j[inrange], s.N)
    # slot rows: source head x = h Gs + g reads slot row b Hslot + x / sdiv
    x_max = h.max() * a.Gs + a.Gs - 1
    assert x_max < a.Hsrc, f"{label}: source head {x_max} >= {a.Hsrc}"
    slot_row_max = (s.B - 1) * s.Hs + x_max // a.sdiv
    assert x_max // a.sdiv < s.Hs
    inside(f"{label} src head", 0, ((s.B - 1) * a.Hsrc + x_max) * s.S * s.D + s.S * s.D, s.B * a.Hsrc * s.S * s.D)
    col_hi = cc.max() * s.CH + s.CH
    inside(f"{label} dst", 0, ((s.B - 1) * s.N + s.N - 1) * a.H * s.D + h.max() * s.D + col_hi, s.B * s.N * a.H * s.D)
    # slot indices read inside one slot row (all unguarded by m < S)
    reads = []
    if a.kind == "long":
        P, TT = s.p, int(round(np.log(RL) / np.log(s.p)))
        LS = min(TT, s.L)
        for l in range(LS, s.L):
            i = c // P ** (l - TT) - shift
            ok = (i >= 0) & (i < s.nrow[l])
            reads.append(s.off[l] + i[ok])
            # every entry of the level whose range meets a written position is looked up
        for l in range(1, LS):
            for s2 in range(P ** (TT - l)):
                i = c * P ** (TT - l) + s2 - shift
                ok = (i >= 0) & (i < s.nrow[l])
                reads.append(s.off[l] + i[ok])
                # the sub-run index r / p^l used by the sums stays inside the run's list
        base = c * RL  # the 4-aligned level-0 block read as vectors: j0 + SH, SH = shift
        vec = a.vec_slots & (c * RL - shift >= 0) & (base + RL <= s.N)
        if a.vec_slots:
            assert (base[vec] % 4 == 0).all()
        reads.append((base[vec][:, None] + np.arange(RL)[None, :]).ravel())
        if a.scatter:
            jj = c[vec] * RL - 1
            reads.append(jj[jj >= 0])
        jn = j[~vec]
        reads.append(jn[(jn >= 0) & (jn < s.N)].ravel())
    elif a.kind == "group_long":
        PL = int(np.log2(s.p))
        j0 = c * 8
        for l in range(1, s.L):
            cnt = 1 if l * PL >= 3 else 1 << (3 - l * PL)
            for e in range(cnt):
                i = (j0 >> (l * PL)) + (0 if cnt == 1 else e)
                ok = i < s.nrow[l]
                reads.append(s.off[l] + i[ok])
        jj = j0[:, None] + np.arange(8)[None, :]
        reads.append(jj[jj < s.N])
    else:  # runs of p (scatter_kernel, gather_bwd_kernel, gather_bwd_group_kernel)
        for l in range(1, s.L):
            i = c // s.pw[l - 1] - shift
            reads.append(s.off[l] + i[i >= 0])
            assert (i < s.nrow[l]).all(), f"{label}: level {l} entry past the level"
        jj = _positions(a.run, c, a.run, shift)
        reads.append(jj[(jj >= 0) & (jj < s.N)])
    reads = np.concatenate([np.asarray(r, np.int64).ravel() for r in reads])
    inside(f"{label} slot index", reads, reads + 1, s.Ptot)
    inside(f"{label} slot row", 0, slot_row_max * s.Ptot + s.Ptot, s.B * s.Hs * s.Ptot)


@pytest.mark.parametrize("name,c,flags", CASES, ids=[x[0] for x in CASES])
def test_scatter_and_gather_bwd_index_math(name, c, flags):
    s = Shape(c, flags)
    _check_run_kernel(s, RunLaunch(s, True, s.Hq, 1, s.Hq, s.Gq), "scatter")
    _check_run_kernel(s, RunLaunch(s, False, s.Hq, 1, s.Hq, s.Gq), "gather_bwd dQ")
    _check_run_kernel(s, RunLaunch(s, False, s.Hkv, s.G // s.Gq, s.Hs, 1), "gather_bwd dK/dV")


def _window_rows(s):
    W = s.P
    while W < 64:
        W += s.P
    return W


@pytest.mark.parametrize("name,c,flags", CASES, ids=[x[0] for x in CASES])
def test_scatter_bwd_index_math(name, c, flags):
    s = Shape(c, flags)
    CPR = 1 << s.cs
    HW = min(s.Hq, 256 // CPR)
    U = s.N + s.P
    W = _window_rows(s)
    gx, gy = -(-U // W), -(-s.Hq // HW)
    hq = (np.arange(gy)[:, None] * HW + np.arange(HW)[None, :]).ravel()
    hq = hq[hq < s.Hq]
    once("scatter_bwd heads", hq, s.Hq)
    assert (hq // s.Gq).max() < s.Hs
    bx = np.arange(gx)
    u0 = bx * W
    nu = np.minimum(U - u0, W)
    assert (nu > 0).all() and (nu % s.P == 0).all(), "a window would straddle two workgroups"
    # level 0: u in [max(u0, 1), min(u0 + nu - 1, N)] reads dout row u - 1 and slot u - 1
    u = np.concatenate([np.arange(a, a + n) for a, n in zip(u0, nu)])
    once("scatter_bwd shifted positions", u, U)
    lvl0 = u[(u >= 1) & (u <= s.N)] - 1
    once("scatter_bwd level-0 entries", lvl0, s.N)
    for l in range(1, s.L):
        epb = W // s.pw[l]
        # windows a closed by workgroup bx: [bx epb, bx epb + nu / p^l); entry i = a - 1
        a_closed = np.concatenate([np.arange(x * epb, x * epb + n // s.pw[l]) for x, n in zip(bx, nu)])
        once(f"scatter_bwd level-{l} windows", a_closed, U // s.pw[l])
        i = a_closed - 1
        assert set(range(s.nrow[l])) <= set(i.tolist()), f"level {l}: an entry's window is never closed"
        # slot prefetches (guarded by 0 <= i < nrows): first window and one past the last
        for wv in (bx * epb, bx * epb + nu // s.pw[l]):
            ii = wv - 1
            ok = (ii >= 0) & (ii < s.nrow[l])
            inside(f"scatter_bwd level-{l} slot", s.off[l] + ii[ok], s.off[l] + ii[ok] + 1, s.Ptot)
    col_hi = (CPR - 1) * s.CH + s.CH
    inside("scatter_bwd dout", 0, ((s.B - 1) * s.N * s.Hq + hq.max()) * s.D + (s.N - 1) * s.Hq * s.D + col_hi,
           s.B * s.N * s.Hq * s.D)
    inside("scatter_bwd dos head", 0, ((s.B - 1) * s.Hq + hq.max()) * s.S * s.D + s.S * s.D, s.B * s.Hq * s.S * s.D)
    inside("scatter_bwd slot row", 0, ((s.B - 1) * s.Hs + (hq.max() // s.Gq)) * s.Ptot + s.Ptot, s.B * s.Hs * s.Ptot)


@pytest.mark.parametrize("name,c,flags", CASES, ids=[x[0] for x in CASES])
def test_pool_score_index_math(name, c, flags):
    s = Shape(c, flags)
    CPR = 1 << s.cs
    Hs3 = [s.Hq, s.Hkv, s.Hkv]
    nslots = sum(Hs3)
    slot1, slot2 = s.Hq, s.Hq + s.Hkv
    HW = max(1, min(nslots, 256 // CPR))
    W = _window_rows(s)
    gx, gy = -(-s.N // W), -(-nslots // HW)
    rowT = s.D + 16 // s.es
    RB = 8
    tile_elems = RB * HW * rowT
    # threads: hs = tid >> cs, cc = tid & (CPR - 1); global head slot gs = by HW + hs
    gs = (np.arange(gy)[:, None] * HW + np.arange(HW)[None, :]).ravel()
    once("pool head slots", gs[gs < nslots], nslots)
    inside("pool LDS rows", 0, ((RB - 1) * HW + HW - 1) * rowT + (CPR - 1) * s.CH + s.CH, tile_elems)
    assert (HW * CPR) <= 256
    bx = np.arange(gx)
    j0 = bx * W
    nrows = np.minimum(s.N - j0, W)
    assert (nrows > 0).all()
    if s.L > 1:
        assert (nrows % s.P == 0).all(), "a pooling window would straddle two workgroups"
        if s.p in (2, 4):  # fixed level-1 closings inside each step of 8 rows
            nr = np.concatenate([np.minimum(n - np.arange(0, n, RB), RB) for n in nrows])
            assert (nr % s.p == 0).all()
    once("pool base rows", np.concatenate([np.arange(a, a + n) for a, n in zip(j0, nrows)]), s.N)
    for t, H in enumerate(Hs3):
        inside(f"pool read t{t}", 0, (((s.B - 1) * s.N + s.N - 1) * H + H - 1) * s.D + CPR * s.CH,
               s.B * s.N * H * s.D)
        for l in range(1, s.L):
            epb = W // s.pw[l]
            rows = np.concatenate([np.arange(x * epb, x * epb + n // s.pw[l]) for x, n in zip(bx, nrows)])
            once(f"pool level-{l} rows t{t}", rows, s.nrow[l])
            prow = (s.off[l] - s.N) + rows
            inside(f"pool pyramid write t{t} l{l}", 0, (((s.B - 1) * s.R + prow.max()) * H + H - 1) * s.D + CPR * s.CH,
                   s.B * s.R * H * s.D)
            if t < 2:  # max-pooled scores of level l: srow[off_l + bx epb + sent]
                inside(f"score write t{t} l{l}", s.off[l] + rows, s.off[l] + rows + 1, s.off[l + 1])
        if t < 2:
            inside(f"score row t{t}", 0, ((s.B - 1) * H + H - 1) * s.Ptot + s.N, s.B * H * s.Ptot)


@pytest.mark.parametrize("name,c,flags", CASES, ids=[x[0] for x in CASES])
def test_selection_workspace_math(name, c, flags):
    s = Shape(c, flags)
    pr = s.problem()
    ws_bytes = lh.lh_workspace_bytes(pr, lh.LH_OP_SELECT)
    BH = s.B * s.Hs
    # candidate lists of (b, selection head) bs at ws + bs Scand, level l at coff[l]
    assert s.coff[s.L] == s.Scand
    inside("select workspace", 0, (BH - 1) * s.Scand + s.Scand, ws_bytes // 4)
    # a level ranks with its keys in LDS (at most 32,768 of them) or, beyond, in one global row
    # of maxsel keys per selection after the lists
    if s.maxsel > 32768:
        inside("select key rows", BH * s.Scand, BH * s.Scand + BH * s.maxsel, ws_bytes // 4)
    # order_kernel: grid ((N + 8191) / 8192, BH); workgroup x owns the window ends [e0, e1) and
    # the level-l entries [e0 // p^l, e1 // p^l): every pyramid entry's slot is written by
    # exactly one workgroup, and its flag index (end - e0) L + (L - 1 - l) stays in [0, 8192 L)
    E = 8192
    gx = -(-s.N // E)
    e0 = np.arange(gx, dtype=np.int64) * E
    e1 = np.minimum(e0 + E, s.N)
    assert e0.max() < 2 ** 31 and (e1 > e0).all()
    for l in range(s.L):
        lo, hi = e0 // s.pw[l], e1 // s.pw[l]
        ids = np.concatenate([np.arange(a, b) for a, b in zip(lo, hi)])
        once(f"order slot entries l{l}", ids, s.nrow[l])
        blk = np.repeat(np.arange(gx), hi - lo)
        x = ((ids + 1) * s.pw[l] - 1 - e0[blk]) * s.L + (s.L - 1 - l)
        inside(f"order flag index l{l}", x, x + 1, E * s.L)
    # the flag scan: 512 threads, thread t owns words [t CW, t CW + CW) clipped to the range's
    # 8192 L / 32 words, so every word is scanned exactly once and ranks fit 16 bits
    NW = E * s.L // 32
    CW = -(-NW // 512)
    own = np.concatenate([np.arange(t * CW, min(t * CW + CW, NW)) for t in range(512)])
    once("order scan words", own, NW)
    assert E * s.L <= 65536
    # every emitted entry gets a distinct rank in [0, S)
    assert s.S <= s.Scand


def _order_by_ranges(N, p, L, lists, replace, E=8192):
    """order_kernel's ranking, restated on the CPU: per range of window ends, the emitted
    entries before it (lower bounds in the sorted lists, less the parents below them in replace
    mode) plus an exclusive scan over the range's (end, level) flags."""
    pw = [p ** l for l in range(L)]
    out = {}
    for e0 in range(0, N, E):
        e1 = min(e0 + E, N)
        r0 = 0
        for l in range(L):
            r0 += int(np.searchsorted(lists[l], e0 // pw[l]))
            if replace and l >= 1:
                r0 -= int(np.searchsorted(lists[l - 1], (e0 // pw[l]) * p)) // p
        flag = np.zeros(E * L, np.int64)
        ent = {}
        for l in range(L):
            a, b = np.searchsorted(lists[l], [e0 // pw[l], e1 // pw[l]])
            for i in lists[l][a:b]:
                i = int(i)
                if replace and l >= 1:
                    c = int(np.searchsorted(lists[l - 1], i * p))
                    if c < len(lists[l - 1]) and lists[l - 1][c] == i * p:
                        continue
                x = ((i + 1) * pw[l] - 1 - e0) * L + (L - 1 - l)
                flag[x] = 1
                ent[x] = (l, i)
        rank = np.cumsum(flag) - flag
        for x, li in ent.items():
            out[li] = r0 + int(rank[x])
    return out


@pytest.mark.parametrize("N,p,L,k,replace,seed", [(4096, 4, 4, 100, False, 1), (4096, 4, 4, 100, True, 2),
                                                  (3000, 5, 3, 40, False, 3), (3000, 5, 3, 40, True, 4),
                                                  (2048, 2, 8, 12, True, 5), (1000, 2, 1, 0, False, 6),
                                                  (8192, 4, 5, 0, False, 7), (5120, 4, 3, 2000, True, 8)])
def test_order_ranges_match_sorted_keys(N, p, L, k, replace, seed):
    """The range-wise ranking equals sorting the emitted entries by key = e L + (L - 1 - l),
    e = (i + 1) p^l - 1, for selections of the structure select_kernel writes (the coarsest
    level whole; each level's candidates the children of the k best of the level above)."""
    rng = np.random.default_rng(seed)
    lists = [None] * L
    lists[L - 1] = np.arange(N // p ** (L - 1))
    for l in range(L - 1, 0, -1):
        npar = min(k, len(lists[l]))
        par = np.sort(rng.choice(lists[l], npar, replace=False))
        lists[l - 1] = (par[:, None] * p + np.arange(p)[None, :]).ravel()
    # the kernel's ranges of 8192 window ends, and short ones that split coarse windows
    got = _order_by_ranges(N, p, L, lists, replace)
    assert got == _order_by_ranges(N, p, L, lists, replace, E=64)
    emitted = []
    for l in range(L):
        child = set(lists[l - 1].tolist()) if (replace and l >= 1) else set()
        for i in lists[l].tolist():
            if i * p in child:
                continue
            emitted.append((((i + 1) * p ** l - 1) * L + (L - 1 - l), l, i))
    emitted.sort()
    want = {(l, i): r for r, (_, l, i) in enumerate(emitted)}
    assert got == want
