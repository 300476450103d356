"""A sweep of small layer chains over the library's dispatch choices (GPU,
against the CPU oracle, OmniCache §3.2-§3.3).

Each case is sized to land on one variant the library picks by shape: the
selection instance by candidates per thread (1, 2, 3 or 4 on the 512- and
1024-thread blocks), the Block Cache compaction in the selection launch, the
similarity tiles by group size, and the attention kernel by head dimension
(16 to 128).  Every case runs a cold and a warm step and applies the same
rules as the other chains (tests/parity.py).
"""
import sys

import pytest
import torch

from oc_synth import small_workload
import paper_2607_23844_amd as oc

from parity import layer_step_parity, shapes, dev_tensor, weights_dev, weights_f64

pytestmark = pytest.mark.gpu

# (what the case reaches, workload arguments)
SWEEP = [
    # token groups of 1200 / 1728 candidates: 512 threads, 3 and 4 per thread
    ("select 512x3", dict(gran="token", F=1, H=40, W=40, C=64, heads=2, head_dim=32, dtype="bf16", r=0.3)),
    ("select 512x4 + ctx", dict(gran="token", F=1, H=48, W=48, C=64, heads=1, head_dim=64, dtype="bf16", r=0.6,
                                n_ctx=5)),
    # 2352 / 3456 candidates: 1024 threads, 3 and 4 per thread
    ("select 1024x3", dict(gran="token", F=1, H=56, W=56, C=32, heads=2, head_dim=16, dtype="bf16", r=0.45)),
    ("select 1024x4", dict(gran="token", F=1, H=64, W=72, C=32, heads=2, head_dim=16, dtype="bf16", r=0.2)),
    ("select 512x3 f32", dict(gran="token", F=1, H=40, W=40, C=32, heads=2, head_dim=16, dtype="f32", r=0.5)),
    # patch-local token groups
    ("token patches k2", dict(gran="token", F=2, H=32, W=32, C=96, heads=3, head_dim=32, dtype="bf16", r=0.5,
                              patch_k=2)),
    ("token patches k3", dict(gran="token", F=1, H=48, W=48, C=128, heads=2, head_dim=64, dtype="bf16", r=0.5,
                              patch_k=3)),
    # Block Cache with the compaction in the selection launch
    ("block 512x3", dict(gran="block", F=4, H=40, W=40, C=32, heads=2, head_dim=16, dtype="bf16", r=0.5)),
    ("block 1024x3", dict(gran="block", F=3, H=56, W=56, C=32, heads=1, head_dim=32, dtype="bf16", r=0.4)),
    ("block patches f32", dict(gran="block", F=3, H=16, W=16, C=48, heads=3, head_dim=16, dtype="f32", r=0.7,
                               patch_k=2)),
    # frame granularities
    ("frame 12", dict(gran="frame", F=12, H=16, W=16, C=64, heads=2, head_dim=32, dtype="bf16", r_frame=0.3,
                      frame_drift=0.3)),
    ("frame patches k4", dict(gran="frame", F=10, H=16, W=16, C=64, heads=2, head_dim=32, dtype="bf16", r_frame=0.4,
                              patch_k=4, frame_drift=0.3)),
    ("frame+token", dict(gran="frame_token", F=8, H=16, W=16, C=64, heads=2, head_dim=32, dtype="bf16", r=0.4,
                         r_frame=0.25, planted=True)),
    # attention head dimensions
    ("head dim 48", dict(gran="token", F=1, H=16, W=16, C=48, heads=1, head_dim=48, dtype="bf16", r=0.5)),
    ("head dim 72", dict(gran="token", F=1, H=32, W=32, C=144, heads=2, head_dim=72, dtype="bf16", r=0.5)),
    ("head dim 80 + ctx", dict(gran="token", F=1, H=32, W=32, C=160, heads=2, head_dim=80, dtype="bf16", r=0.5,
                               n_ctx=9)),
    ("head dim 96", dict(gran="token", F=1, H=32, W=32, C=96, heads=1, head_dim=96, dtype="bf16", r=0.5)),
    ("head dim 128", dict(gran="token", F=1, H=24, W=24, C=256, heads=2, head_dim=128, dtype="bf16", r=0.5)),
]


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("case", range(len(SWEEP)), ids=[c[0].replace(" ", "_") for c in SWEEP])
def test_sweep_chain(case):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    name, kw = SWEEP[case]
    wl = small_workload(n_steps=2, seed=300 + case, **kw)
    _say(f"sweep case {case} ({name}): {kw}")
    sh, cf, osh, ocf = shapes(wl)
    dev = torch.device("cuda:0")
    ws = oc.workspace(sh, cf, dev)
    cache = oc.LayerCache(sh, dev)
    ctx_dev = dev_tensor(wl, wl.ctx) if wl.n_ctx else None
    ctx64 = wl.f64(wl.ctx) if wl.n_ctx else None
    W, W64 = weights_dev(wl), weights_f64(wl)
    ora, valid = None, False
    for s in range(2):
        res, st = layer_step_parity(wl, wl.steps[s], sh, cf, osh, ocf, cache, ws, ora, valid, ctx_dev, ctx64, W,
                                    W64, case=f"sweep {name}")
        _say(f"  step {s}: {st}")
        ora, valid = res.y, True
        assert cache.valid == 1 and cache.step == s + 1
