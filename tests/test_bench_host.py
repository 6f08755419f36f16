"""Host-side checks of bench.py: the algorithmic work behind every roofline figure, and the
one-GPU contract. No GPU is touched."""
from __future__ import annotations

import os
import subprocess
import sys

import pytest

import paper_2605_06554_amd as lh
import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402

# Algorithmic work per layer call, counted by hand from the stage definitions (every stage
# boundary materialised; bf16 elements): memory stages in GB (pool+score, select, gather,
# scatter, scatter adjoint, gather+pool adjoint) and SDPA in TFLOP (forward 2 GEMMs, backward 4).
EXPECTED = {
    "c2": ((0.270, 0.004, 0.333, 0.123, 0.123, 0.368), 0.754, 1.508),
    "c3": ((4.323, 0.051, 3.725, 1.694, 1.694, 5.083), 23.5, 47.0),
    "c4": ((4.347, 0.066, 2.668, 2.592, 2.592, 4.555), 24.1, 48.3),
    "c5": ((17.355, 0.113, 2.944, 4.786, 4.786, 14.357), 58.8, 117.6),
}
MEM_STAGES = ("pool_score", "select", "gather", "scatter", "scatter_bwd", "gather_bwd")


@pytest.mark.parametrize("name", sorted(EXPECTED))
def test_stage_work_matches_hand_count(name):
    cfg = workloads.CONFIGS[name]
    pr = lh.problem(cfg.B, cfg.N, cfg.Hq, cfg.Hkv, cfg.D, cfg.p, cfg.L, cfg.k, lh.LH_BF16)
    S, Ptot = lh.lh_subseq_len(pr), lh.lh_pyramid_rows(pr)
    work = bench.stage_work(pr, S, Ptot, 2)
    mem, fwd, bwd = EXPECTED[name]
    for stage, gb in zip(MEM_STAGES, mem):
        bound, amount = work[stage]
        assert bound == "hbm"
        assert amount / 1e9 == pytest.approx(gb, abs=1.5e-3), stage
    assert work["sdpa_fwd"] == ("mfma", pytest.approx(fwd * 1e12, rel=5e-3))
    assert work["sdpa_bwd"] == ("mfma", pytest.approx(bwd * 1e12, rel=5e-3))


def test_sdpa_flops_are_causal_pair_counts():
    """2 GEMMs of 2 D flops per causal (query, key) pair forward, 4 backward."""
    pr = lh.problem(1, 1024, 2, 2, 64, 4, 3, 128, lh.LH_BF16)
    S = lh.lh_subseq_len(pr)
    work = bench.stage_work(pr, S, lh.lh_pyramid_rows(pr), 2)
    pairs = sum(m + 1 for m in range(S)) * 2  # two heads
    assert work["sdpa_fwd"][1] == 2 * 2 * 64 * pairs
    assert work["sdpa_bwd"][1] == 4 * 2 * 64 * pairs


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=300, env={**os.environ, "HIP_VISIBLE_DEVICES": ""})
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""
