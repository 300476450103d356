"""The hand-worked goldens of tests/golden/ run through the HIP library.

The golden inputs are small integers (exact in fp32 and bf16) chosen so
that every tie of the worked examples is an exact tie in any arithmetic:
the tied similarities come from the same dot product and the same norms.
So the library must reproduce, bit for bit, every best-match index (exact
ties resolved to the smallest representative, a zero-norm item matched with
similarity 0, a best match of 0 beside a -1), the cached set at every ratio
of the file, kept_idx, and both restore maps (valid cache and the cold
"matched" policy) — OmniCache §3.2.1 (Block Cache), §3.2.2 (Frame Cache),
§3.2.3 (Token Cache).  The channel count is padded with zeros to the
library's multiple of 8, which leaves every cosine unchanged.
"""
import sys

import numpy as np
import pytest
import torch

from oc_synth import bf16_bits, small_workload
import goldens
from oracle import oc_oracle as O
import paper_2607_23844_amd as oc

from parity import TOL, RAW_TOL, dev_tensor, rel_err, to_f64, weights_dev, weights_f64

pytestmark = pytest.mark.gpu

CASES = [("token_4x4_worked.json", "token", "r"), ("frame_6x2x2_worked.json", "frame", "r_frame"),
         ("block_2x2x4_worked.json", "block", "r")]
C_PAD = 8


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _golden(name):
    g, x = goldens.load(name, np.float32)
    F, N, C = x.shape
    xp = np.zeros((F, N, C_PAD), dtype=np.float32)
    xp[:, :, :C] = x
    return g, F, g["H"], g["W"], xp


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    oc.lib()


def _cfg(gran, key, ratio, cold="matched"):
    return oc.Cfg(gran, ratio if key == "r" else 0.0, ratio if key == "r_frame" else 0.0, 1, cold)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("name,gran,key", CASES, ids=[c[1] for c in CASES])
def test_golden_decisions_bit_exact(name, gran, key, dtype):
    g, F, H, W, x32 = _golden(name)
    _say(f"golden {name} {dtype}")
    wl = small_workload(gran, F=F, H=H, W=W, C=C_PAD, heads=1, head_dim=16, dtype=dtype, seed=3)
    x_np = bf16_bits(x32) if dtype == "bf16" else x32
    sh = oc.Shape(F, H, W, C_PAD, 1, 16, 0, dtype)
    x = dev_tensor(wl, x_np)
    expect_max = np.array([goldens.value(s) for s in g["node_max"]])
    for ratio, cached in g["cached"].items():
        cf = _cfg(gran, key, float(ratio))
        ws = oc.workspace(sh, cf, x.device)
        nm, ni = oc.match(x, sh, cf, ws)
        kept, cidx, rmap = oc.select(nm, ni, sh, cf, ws)
        torch.cuda.synchronize()
        assert nm.shape[0] == 1
        np.testing.assert_array_equal(ni[0].cpu().numpy(), g["node_idx"])
        d = np.abs(nm[0].cpu().numpy().astype(np.float64) - expect_max)
        assert d.max() <= 2e-6, d
        got = sorted({int(p) // (H * W) if gran == "frame" else (int(p) % (H * W) if gran == "block" else int(p))
                      for p in cidx.cpu().numpy()})
        assert got == cached, f"ratio {ratio}: cached {got}, expected {cached}"
    # a cold "matched" step, then a warm step: kept rows and both maps
    W_dev, W64 = weights_dev(wl), weights_f64(wl)
    osh = O.LayerShape(F, H, W, C_PAD, 1, 16)
    x64 = wl.f64(x_np).reshape(F, H * W, C_PAD)
    for mk in (k for k in g if k.startswith("r0")):
        ratio = float(mk[1:])
        cf = _cfg(gran, key, ratio)
        ocf = O.CacheCfg(gran, r=cf.r, r_frame=cf.r_frame)
        ws = oc.workspace(sh, cf, x.device)
        cache = oc.LayerCache(sh, x.device)
        prev = None
        for valid, mapkey in ((False, "restore_map_cold_matched"), (True, "restore_map_valid_cache")):
            y, _, tr = oc.layer_cached(x, W_dev, cache, sh, cf, ws=ws, trace=True)
            torch.cuda.synchronize()
            np.testing.assert_array_equal(tr["kept_idx"].cpu().numpy(), g[mk]["kept_idx"])
            np.testing.assert_array_equal(tr["restore_map"].cpu().numpy(), g[mk][mapkey])
            res = O.layer_step(x64, None, W64, osh, ocf, prev, valid)
            yg = to_f64(y).reshape(res.y.shape)
            err, raw = rel_err(yg, res.y, dtype), rel_err(yg, res.y)
            _say(f"  {mk} {mapkey}: output error {err:.3g} (raw {raw:.3g})")
            assert err <= TOL[dtype] and raw <= RAW_TOL[dtype]
            prev = res.y


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_golden_frame_patches_bit_exact(dtype):
    """Frame Cache on 2x2 patches (§3.3) on the hand-worked 4-frame example:
    per-patch best matches and selections at both ratios, the frame-major
    kept rows with sequences of 16/4/16/12 and 16/0/16/0 tokens (frames that
    keep nothing), and both restore maps, bit for bit."""
    g, x = goldens.load("frame_patch_4x4x4_worked.json", np.float32)
    F, H, W, C, k = g["F"], g["H"], g["W"], g["C"], g["patch_k"]
    xp = np.zeros((F, H * W, C_PAD), dtype=np.float32)
    xp[:, :, :C] = x
    wl = small_workload("frame", F=F, H=H, W=W, C=C_PAD, heads=1, head_dim=16, dtype=dtype, seed=4)
    x_np = bf16_bits(xp) if dtype == "bf16" else xp
    sh = oc.Shape(F, H, W, C_PAD, 1, 16, 0, dtype)
    x = dev_tensor(wl, x_np)
    for ratio, cached in g["cached"].items():
        cf = oc.Cfg("frame", 0.0, float(ratio), k, "matched")
        ws = oc.workspace(sh, cf, x.device)
        nm, ni = oc.match(x, sh, cf, ws)
        kept, cidx, rmap = oc.select(nm, ni, sh, cf, ws)
        torch.cuda.synchronize()
        assert nm.shape[0] == k * k
        for gi, gg in enumerate(g["groups"]):
            np.testing.assert_array_equal(ni[gi].cpu().numpy(), gg["node_idx"])
            d = np.abs(nm[gi].cpu().numpy().astype(np.float64) - np.array([goldens.value(s) for s in gg["node_max"]]))
            assert d.max() <= 2e-6, d
        assert len(cidx) == len(cached) * (H // k) * (W // k)
        tiles = set()
        for p in cidx.cpu().numpy():
            f, n = divmod(int(p), H * W)
            y, xx = divmod(n, W)
            tiles.add(f * H * W + (y // 2) * 2 * W + (xx // 2) * 2)
        assert tiles == set(cached)
    W_dev, W64 = weights_dev(wl), weights_f64(wl)
    osh = O.LayerShape(F, H, W, C_PAD, 1, 16)
    x64 = wl.f64(x_np).reshape(F, H * W, C_PAD)
    for mk in ("r0.25", "r0.5"):
        cf = oc.Cfg("frame", 0.0, float(mk[1:]), k, "matched")
        ocf = O.CacheCfg("frame", r_frame=cf.r_frame, patch_k=k)
        ws = oc.workspace(sh, cf, x.device)
        cache = oc.LayerCache(sh, x.device)
        prev = None
        for valid, mapkey in ((False, "restore_map_cold_matched"), (True, "restore_map_valid_cache")):
            y, _, tr = oc.layer_cached(x, W_dev, cache, sh, cf, ws=ws, trace=True)
            torch.cuda.synchronize()
            np.testing.assert_array_equal(tr["kept_idx"].cpu().numpy(), g[mk]["kept_idx"])
            np.testing.assert_array_equal(tr["restore_map"].cpu().numpy(), g[mk][mapkey])
            res = O.layer_step(x64, None, W64, osh, ocf, prev, valid)
            assert [len(s) for s in res.sequences] == g[mk]["sequence_lengths"]
            yg = to_f64(y).reshape(res.y.shape)
            err, raw = rel_err(yg, res.y, dtype), rel_err(yg, res.y)
            _say(f"  frame patches {mk} {mapkey}: output error {err:.3g} (raw {raw:.3g})")
            assert err <= TOL[dtype] and raw <= RAW_TOL[dtype]
            prev = res.y
