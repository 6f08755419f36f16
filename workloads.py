"""Seeded synthetic workloads for the Lighthouse attention hot path.

This module only draws inputs; it holds none of the method's arithmetic. The GPU path, the
oracle and the benchmark all take their inputs from here.

The paper's workloads (a 530M Llama-style model on C4, and an unspecified single-layer latency
bench: B=1, H=8, d=128, bf16, N from 8K to 512K; Sec. 6) are not available. These synthetic
inputs stand in for them at the same shape class. Recipe (fixed per config):
  * a generator seeded with 1000 + config number (a torch.Generator on the requested device,
    so device-generated inputs are reproducible but differ from host-generated ones);
  * draw order: Q, K, V, dO (all standard normal, float32), then the structure draws;
  * structure is applied in float32 and the result is cast once (round to nearest even) to
    the config dtype.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace

import torch


@dataclass(frozen=True)
class Config:
    name: str
    B: int
    N: int
    Hq: int
    Hkv: int
    D: int
    p: int
    L: int
    k: int
    dtype: str            # "fp32" | "bf16"
    seed: int
    structure: str = "iid"     # "iid" | "spikes" | "subspace"
    spike_frac: float = 0.0
    spike_scale: float = 8.0
    rank: int = 64
    noise: float = 0.1
    flags: int = 0
    notes: str = field(default="", compare=False)

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "fp32" else torch.bfloat16


# The five configurations of the benchmark contract (one Lighthouse layer each).
CONFIGS = {
    "c1": Config("c1", 1, 1024, 2, 2, 64, 4, 3, 128, "fp32", 1001,
                 notes="iid N(0,1); oracle runs in seconds"),
    "c2": Config("c2", 1, 16384, 16, 16, 128, 4, 4, 2048, "bf16", 1002, "spikes", 0.01,
                 notes="1% of key positions scaled x8 in every head"),
    "c3": Config("c3", 2, 65536, 32, 32, 128, 4, 4, 4096, "bf16", 1003, "subspace",
                 notes="Q,K in a rank-64 per-head subspace plus N(0,0.1) noise"),
    "c4": Config("c4", 1, 262144, 32, 8, 128, 4, 5, 4096, "bf16", 1004, "spikes", 0.005,
                 notes="GQA 32/8; 0.5% of key positions scaled x8 in every KV head"),
    "c5": Config("c5", 1, 1048576, 16, 16, 128, 4, 6, 8192, "bf16", 1005,
                 notes="iid N(0,1); ~4 GB per tensor"),
}

# One GPU's share of a configuration sharded by KV group (G query heads and their KV head per
# GPU, no communication inside the layer): c4 over 8 GPUs.
SHARD_CONFIGS = {
    "c4-kv1": Config("c4-kv1", 1, 262144, 4, 1, 128, 4, 5, 4096, "bf16", 1004, "spikes", 0.005,
                     notes="one GPU's share of c4 over 8 GPUs: one KV head and its 4 query heads"),
}

# Small shapes for parity tests: several tiles and a ragged tail, oracle in seconds.
TEST_CONFIGS = {
    # S = 64 + 256 + 1024 + 1024 = 2368 (ragged against 64/128/256-row tiles)
    "t_gqa": Config("t_gqa", 1, 4096, 4, 2, 128, 4, 4, 256, "bf16", 2001, "spikes", 0.01),
    # B = 2, D = 64, p = 2: S = 128 + 2*(2*96) = 512? computed by the library; fp32
    "t_f32": Config("t_f32", 2, 1024, 2, 1, 64, 2, 4, 96, "fp32", 2002),
    # p = 3 (non power of two pooling), bf16
    "t_p3": Config("t_p3", 1, 2187, 2, 2, 64, 3, 3, 100, "bf16", 2003),
    # L = 1: plain causal SDPA on N rows
    "t_l1": Config("t_l1", 1, 777, 2, 2, 128, 4, 1, 0, "bf16", 2004),
    # k = 0: only the coarsest level
    "t_k0": Config("t_k0", 1, 1024, 2, 2, 128, 4, 3, 0, "bf16", 2005),
    # stratified selection (flag bit 1): levels 2 and 1 rank 4096 and 3000 candidates in chunks
    # of 2048, S = 4096 + 3000 + 3000
    "t_strat": Config("t_strat", 1, 16384, 2, 1, 64, 2, 3, 1500, "bf16", 2006, "spikes", 0.01, flags=2),
    # L = 2 with N = 4 * 257: the last run of p^2 positions is partial; Ptot = 1285 (odd)
    "t_l2": Config("t_l2", 1, 1028, 2, 2, 64, 4, 2, 64, "bf16", 2007),
    # L = 2, N = 4 * 257, two query heads per KV head: the dK / dV gather adjoint sums a
    # group over runs of 8 positions, and its last run is partial
    "t_l2g": Config("t_l2g", 1, 1028, 4, 2, 64, 4, 2, 64, "bf16", 2012),
    # p = 3 and p = 5 with two query heads per KV head: the runs-of-p grouped adjoint (p = 3)
    # and the generic scatter and adjoint kernels for p > 4
    "t_p3g": Config("t_p3g", 1, 999, 4, 2, 64, 3, 3, 40, "bf16", 2013),
    "t_p5g": Config("t_p5g", 1, 1000, 4, 2, 64, 5, 3, 30, "bf16", 2014),
    # L = 8, the deepest pyramid the kernels are instantiated for (p = 2, N = 2048)
    "t_l8": Config("t_l8", 1, 2048, 2, 1, 64, 2, 8, 12, "bf16", 2015),
    # p = 2, L = 5, N = 112: Ptot = 217 (odd), three query heads per KV head
    "t_g3": Config("t_g3", 1, 112, 3, 1, 64, 2, 5, 5, "bf16", 2008),
    # dK / dV gather adjoint over runs of 8 positions with a whole wave or more per run (p = 4,
    # 2 or 4 query heads per KV head, the unpacked launch of the c4 layer): G = 4 with spiked
    # keys (Ptot = 5440); a partial last run (N = 4 * 257); fp32; two workgroups per run
    # (32 KV heads, 512 threads of work per run)
    "t_grp4": Config("t_grp4", 1, 4096, 16, 4, 128, 4, 4, 128, "bf16", 2016, "spikes", 0.01),
    "t_grp_tail": Config("t_grp_tail", 2, 1028, 8, 4, 128, 4, 2, 64, "bf16", 2017),
    "t_grp_f32": Config("t_grp_f32", 2, 1024, 8, 4, 64, 4, 3, 32, "fp32", 2018),
    "t_grp_wide": Config("t_grp_wide", 1, 256, 64, 32, 128, 4, 3, 8, "bf16", 2019),
    # one selection per KV group (flag bit 2): G = 2, p = 4; G = 3, p = 2; G = 4 in fp32
    "t_gqs": Config("t_gqs", 1, 4096, 4, 2, 128, 4, 4, 256, "bf16", 2009, "spikes", 0.01, flags=4),
    "t_gqs3": Config("t_gqs3", 1, 2048, 6, 2, 64, 2, 5, 40, "bf16", 2010, flags=4),
    "t_gqs_f32": Config("t_gqs_f32", 1, 1024, 4, 1, 64, 4, 3, 64, "fp32", 2011, flags=4),
}


def scaled(cfg: Config, **kw) -> Config:
    """A copy of cfg with some fields replaced (e.g. a shorter N for a quick run)."""
    return replace(cfg, **kw)


def make_inputs(cfg: Config, device: str = "cpu", with_grad: bool = True):
    """Draws q [B,N,Hq,D], k, v [B,N,Hkv,D] and dout [B,N,Hq,D] in the config dtype."""
    g = torch.Generator(device=device)
    g.manual_seed(cfg.seed)
    f32 = dict(dtype=torch.float32, device=device, generator=g)
    q = torch.randn(cfg.B, cfg.N, cfg.Hq, cfg.D, **f32)
    k = torch.randn(cfg.B, cfg.N, cfg.Hkv, cfg.D, **f32)
    v = torch.randn(cfg.B, cfg.N, cfg.Hkv, cfg.D, **f32)
    dout = torch.randn(cfg.B, cfg.N, cfg.Hq, cfg.D, **f32) if with_grad else None
    if cfg.structure == "spikes":
        n_spk = int(round(cfg.spike_frac * cfg.N))
        pos = torch.randperm(cfg.N, generator=g, device=device)[:n_spk]
        k[:, pos] *= cfg.spike_scale
    elif cfg.structure == "subspace":
        # per head h: an orthonormal basis U_h [D, rank] shared by Q and K of that head
        for h in range(cfg.Hq):
            a = torch.randn(cfg.D, cfg.rank, **f32)
            U, _ = torch.linalg.qr(a.cpu())
            U = U.to(device)
            zq = torch.randn(cfg.B, cfg.N, cfg.rank, **f32)
            zk = torch.randn(cfg.B, cfg.N, cfg.rank, **f32)
            q[:, :, h, :] = zq @ U.T + cfg.noise * torch.randn(cfg.B, cfg.N, cfg.D, **f32)
            if h < cfg.Hkv:
                k[:, :, h, :] = zk @ U.T + cfg.noise * torch.randn(cfg.B, cfg.N, cfg.D, **f32)
    dt = cfg.torch_dtype
    out = dict(q=q.to(dt), k=k.to(dt), v=v.to(dt))
    out["dout"] = dout.to(dt) if dout is not None else None
    if cfg.structure == "spikes":
        out["spikes"] = pos.cpu()
    return out


def spike_positions(cfg: Config, device: str = "cpu"):
    """Replays the draws of make_inputs up to the spike positions (without keeping tensors)."""
    return make_inputs(cfg, device, with_grad=True).get("spikes")
