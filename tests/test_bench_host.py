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
    cfg = oc.Cfg("token", r=0.5, patch_k=1)
    pl = oc.plan(shape, cfg)
    assert (pl.n_kept, pl.n_seq, pl.seq_len) == (2048, 1, 2048)
    assert (pl.n_groups, pl.n_src_max, pl.n_dst_max) == (1, 3072, 1024)
    w = bench.stage_work(shape, cfg, pl, 333)
    rows, C, hd = 2048 + 333, 1536, 24 * 64
    assert w["proj_qkv"][0] == 2.0 * rows * C * 3 * hd == 33704902656.0
    assert w["proj_qkv"][1] == 2.0 * (rows * C + 3 * hd * C + 3 * rows * hd)   # x rows, weights, Q K V out
    assert w["flash"] == (4.0 * rows * rows * hd, 2.0 * 4 * rows * hd)          # Q K^T and P V; Q K V in, O out
    assert w["proj_out"][0] == 2.0 * rows * hd * C
    assert w["match"][0] == 2.0 * 3072 * 1024 * C                              # every candidate x every rep
    assert w["inv_norm"][1] == 4096 * C * 2.0 + 4096 * 4.0                     # read x (bf16), one norm per token
    assert w["gather"][1] == 2.0 * 2048 * C * 2.0
    # the bound is the resource with the longer ideal time
    assert bench.roofline_of(*w["flash"], 50.0)["bound"] == "mfma"
    assert bench.roofline_of(*w["inv_norm"], 7.0)["bound"] == "hbm"
    r = bench.roofline_of(*w["flash"], 50.0)
    assert r["achieved"] == pytest.approx(w["flash"][0] / 50e-6 / 1e12, rel=1e-3)


def test_stage_work_counts_sequences_apart_without_context():
    # Block Cache on a Latte-like temporal layer: 128 retained positions, each
    # a sequence of its 16 frames; attention work is per sequence, and the
    # block descriptors are F*C long
    shape = oc.Shape(16, 16, 16, 1152, 16, 72, 0, "bf16")
    cfg = oc.Cfg("block", r=0.5, patch_k=1)
    pl = oc.plan(shape, cfg)
    assert (pl.n_seq, pl.seq_len, pl.n_kept) == (128, 16, 2048)
    w = bench.stage_work(shape, cfg, pl, 0)
    assert w["flash"][0] == 4.0 * 128 * 16 * 16 * 16 * 72
    assert w["proj_qkv"][0] == 2.0 * 2048 * 1152 * 3 * 16 * 72
    assert w["match"][0] == 2.0 * 192 * 64 * 16 * 1152
    assert bench.roofline_of(*w["match"], 10.0)["bound"] == "hbm"              # 48 flop per byte
