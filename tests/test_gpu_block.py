"""A spatial + temporal block with all three caches (oc_block_cached) at the
paper's operating points: Latte 30/40/20 and SVD-XT 50/40/50 (r_f / r_b /
r_t, OmniCache §4.2), several denoising steps, each layer carrying its own
cache.  Each layer is checked against the oracle on its exact input: the
spatial layer on x, the temporal layer on the h the library stored; the
residual h = x + y_spatial is checked bit for bit against the same fp32 sum
rounded to bf16 on the host."""
import sys

import numpy as np
import pytest
import torch

from oc_synth import bf16_bits, make_workload
from oracle import oc_oracle as O
import paper_2607_23844_amd as oc

from parity import (check_layer_step, check_layer_step_sampled, dev_tensor, weights_dev, weights_f64)

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    oc.lib()


def _bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def block_chain(name, n_steps, n_sample=None, seed=31):
    wl = make_workload(name, n_steps)
    sh = oc.Shape(wl.F, wl.H, wl.W, wl.C, wl.heads, wl.head_dim, 0, "bf16")
    cs_cfg = oc.Cfg(wl.gran, wl.r, wl.r_frame, wl.patch_k, "matched")
    ct_cfg = oc.Cfg("block", wl.extra["r_block"], 0.0, wl.extra["block_patch_k"], "matched")
    osh = O.LayerShape(wl.F, wl.H, wl.W, wl.C, wl.heads, wl.head_dim)
    ocs = O.CacheCfg(wl.gran, wl.r, wl.r_frame, wl.patch_k, "matched")
    oct_ = O.CacheCfg("block", wl.extra["r_block"], 0.0, wl.extra["block_patch_k"], "matched")
    dev = torch.device("cuda:0")
    Ws, Wt = weights_dev(wl), weights_dev(wl, wl.t_weights)
    W64s, W64t = weights_f64(wl), weights_f64(wl, wl.t_weights)
    c_s, c_t = oc.LayerCache(sh, dev), oc.LayerCache(sh, dev)
    h = torch.empty((wl.F, wl.N, wl.C), dtype=torch.bfloat16, device=dev)
    ws = oc.block_workspace(sh, cs_cfg, ct_cfg, dev)
    rng = np.random.default_rng(seed)
    pos = None if n_sample is None else np.sort(rng.choice(wl.F * wl.N, n_sample, replace=False))
    ora_s = ora_t = None
    valid = False
    for s in range(n_steps):
        _say(f"  step {s} of {name}: spatial {wl.gran} r_t={wl.r} r_f={wl.r_frame} k={wl.patch_k}, "
             f"temporal block r_b={wl.extra['r_block']} k={wl.extra['block_patch_k']}")
        x = dev_tensor(wl, wl.steps[s])
        y, h, trs, trt = oc.block_cached(x, Ws, Wt, c_s, c_t, sh, cs_cfg, ct_cfg, h=h, ws=ws, trace=True)
        torch.cuda.synchronize()
        assert (c_s.valid, c_s.step, c_t.valid, c_t.step) == (1, s + 1, 1, s + 1)
        # the residual: fp32 sum of the two bf16 tensors, rounded to bf16
        expect = bf16_bits(wl.to_f32(wl.steps[s]).reshape(-1) + wl.to_f32(_bits(c_s.y)).reshape(-1))
        assert np.array_equal(_bits(h).reshape(-1), expect), "residual h differs from bf16(x + y_spatial)"
        h64 = wl.f64(_bits(h)).reshape(wl.F, wl.N, wl.C)
        x64 = wl.f64(wl.steps[s])
        if pos is None:
            rs, sts = check_layer_step(x64, None, W64s, osh, ocs, ora_s, valid, c_s.y, None, trs, "bf16")
            rt, stt = check_layer_step(h64, None, W64t, osh, oct_, ora_t, valid, c_t.y, None, trt, "bf16")
            ora_s, ora_t = rs.y, rt.y
        else:
            ora_s, sts = check_layer_step_sampled(x64, W64s, osh, ocs, valid, c_s.y, trs, pos, ora_s, "bf16")
            ora_t, stt = check_layer_step_sampled(h64, W64t, osh, oct_, valid, c_t.y, trt, pos, ora_t, "bf16")
        _say(f"    spatial {sts}\n    temporal {stt}")
        valid = True


def test_latte_block_chain():
    """Latte-like block (16 frames of 16x16, C=1152, 16 x 72): spatial Frame +
    Token Cache at r_f = 0.3, r_t = 0.2, temporal Block Cache at r_b = 0.4,
    four steps, outputs of both layers checked in full."""
    block_chain("latte_block", 4)


def test_svdxt_block_sampled_chain():
    """SVD-XT-like block (25 frames of 72x128, C=320, 5 x 64) at r_f = 0.5,
    r_b = 0.4, r_t = 0.5, patch-local 4x4 matching for tokens and blocks:
    decisions and maps in full, outputs at 256 sampled positions."""
    block_chain("svdxt_block", 2, n_sample=256)
