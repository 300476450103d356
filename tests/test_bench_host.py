"""Host-side parts of bench.py (no GPU): the one-GPU contract and the
algorithmic work per launch that the roofline figures divide by."""
import os
import subprocess
import sys

import pytest

import bench
import paper_2607_23844_amd as oc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("n", [2, 8])
def test_more_than_one_gpu_is_refused(n):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", str(n)], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_stage_work_at_the_sd3_shape():
    # 64x64 image tokens + 333 text tokens, C = 1536, 24 heads x 64, r = 0.5:
    # 2048 of the 4096 image tokens are retained (the 1024 window
    # representatives are always kept, 1024 of the 3072 candidates too)
    shape = oc.Shape(1, 64, 64, 1536, 24, 64, 333, "bf16")
    pl = oc.plan(shape, oc.Cfg("token", r=0.5, patch_k=1))
    assert (pl.n_kept, pl.n_seq, pl.seq_len) == (2048, 1, 2048)
    assert (pl.n_groups, pl.n_src_max, pl.n_dst_max) == (1, 3072, 1024)
    w = bench.stage_work(shape, pl, 333)
    rows, C, hd = 2048 + 333, 1536, 24 * 64
    assert w["proj_qkv"] == ("mfma", 2.0 * rows * C * 3 * hd) and w["proj_qkv"][1] == 33704902656.0
    assert w["flash"] == ("mfma", 4.0 * rows * rows * hd)          # Q K^T and P V over one sequence
    assert w["proj_out"] == ("mfma", 2.0 * rows * hd * C)
    assert w["match"] == ("mfma", 2.0 * 3072 * 1024 * C)           # every candidate against every representative
    assert w["inv_norm"] == ("hbm", 4096 * C * 2.0 + 4096 * 4.0)   # read x (bf16), write one norm per token
    assert w["gather"] == ("hbm", 2.0 * 2048 * C * 2.0)


def test_stage_work_counts_sequences_apart_without_context():
    # Block Cache on a Latte-like temporal layer: 128 retained positions, each
    # a sequence of its 16 frames; attention work is per sequence
    shape = oc.Shape(16, 16, 16, 1152, 16, 72, 0, "bf16")
    pl = oc.plan(shape, oc.Cfg("block", r=0.5, patch_k=1))
    assert (pl.n_seq, pl.seq_len, pl.n_kept) == (128, 16, 2048)
    w = bench.stage_work(shape, pl, 0)
    assert w["flash"][1] == 4.0 * 128 * 16 * 16 * 16 * 72
    assert w["proj_qkv"][1] == 2.0 * 2048 * 1152 * 3 * 16 * 72
