"""oc_layer_cached_static (the entry point for callers that cannot
allocate) against oc_layer_cached with a caller workspace: four layers in
a row through the library's static scratch, each smaller than the one
before (so it runs over the previous call's leftover scratch contents),
each for a cold and a warm step.  Same kernels on the same inputs: outputs,
context outputs and decision traces must be bit-identical."""
import sys

import pytest
import torch

from oc_synth import make_workload, small_workload
import paper_2607_23844_amd as oc

from parity import dev_tensor, shapes, weights_dev

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _same(a, b):
    if a.dtype in (torch.bfloat16, torch.float16):
        return torch.equal(a.view(torch.int16), b.view(torch.int16))
    return torch.equal(a, b)


def test_static_scratch_matches_workspace_entry_point():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    dev = torch.device("cuda:0")
    # the SD3-like layer (57 MiB of scratch), then the smaller Latte-like
    # spatial Frame Cache layer (41 MiB), then a small Frame+Token Cache
    # layer, then a small two-level Token Cache layer (patches of 4 x 4, then
    # the whole frame)
    layers = [(make_workload("sd3_1024", 2), {}), (make_workload("latte_spatial", 2), {}),
              (small_workload("frame_token", F=7, H=8, W=8, C=64, heads=2, head_dim=32, dtype="bf16", r_frame=0.3,
                              planted=True, n_steps=2, seed=8), {}),
              (small_workload("token", F=1, H=16, W=16, C=64, heads=2, head_dim=32, dtype="bf16", n_steps=2, seed=9),
               dict(r=0.25, patch_k=4, coarse_k=1, r_coarse=0.25))]
    for wl, kw in layers:
        sh, cf, _, _ = shapes(wl, **kw)
        need = oc.plan(sh, cf).workspace_bytes
        _say(f"{wl.name}: scratch {need / 2**20:.1f} MiB of {oc.static_scratch_bytes() / 2**20:.0f}")
        assert need <= oc.static_scratch_bytes()
        W = weights_dev(wl)
        ctx = dev_tensor(wl, wl.ctx) if wl.n_ctx else None
        ws = oc.workspace(sh, cf, dev)
        c_ws, c_st = oc.LayerCache(sh, dev), oc.LayerCache(sh, dev)
        for s in range(2):
            x = dev_tensor(wl, wl.steps[s])
            y1, yc1, t1 = oc.layer_cached(x, W, c_ws, sh, cf, ctx=ctx, ws=ws, trace=True)
            y2, yc2, t2 = oc.layer_cached_static(x, W, c_st, sh, cf, ctx=ctx, trace=True)
            torch.cuda.synchronize()
            assert _same(y1, y2), f"{wl.name} step {s}: outputs differ"
            if ctx is not None:
                assert _same(yc1, yc2), f"{wl.name} step {s}: context outputs differ"
            keys = ["node_max", "node_idx", "kept_idx", "cached_idx", "restore_map"]
            if cf.gran == "frame_token":        # the frame stage is traced for Frame+Token only
                keys += ["frame_max", "frame_idx", "pairs"]
            for k in keys:
                assert _same(t1[k], t2[k]), f"{wl.name} step {s}: trace {k} differs"
            assert (c_ws.valid, c_ws.step) == (c_st.valid, c_st.step) == (1, s + 1)
            _say(f"  step {s}: bit-identical ({t1['kept_idx'].numel()} retained tokens)")
