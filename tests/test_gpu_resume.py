"""Checkpoint and resume of a cached chain (the layer cache carried across
denoising steps, OmniCache §3.1-§3.2: a cached step restores positions from
the previous step's layer output).  The whole state a chain carries is the
layer cache: its output buffer y, its valid flag and its step count.  A chain
that is stopped after two steps, whose cache is written to a file, read back
into a fresh cache (and a fresh workspace), and continued, must give the
uninterrupted chain's outputs bit for bit, for every granularity and at the
SD3-sized layer the benchmark times."""
import sys

import pytest
import torch

from oc_synth import make_workload, small_workload
import paper_2607_23844_amd as oc

from parity import dev_tensor, shapes, weights_dev

pytestmark = pytest.mark.gpu

N_STEPS = 4
STOP_AFTER = 2


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    oc.lib()


def _run(wl, sh, cf, W, xs, ctx, cache, ws, steps):
    out = []
    for s in steps:
        y, y_ctx, _ = oc.layer_cached(xs[s], W, cache, sh, cf, ctx=ctx, ws=ws)
        torch.cuda.synchronize()
        out.append((y.view(torch.int16).clone(), None if y_ctx is None else y_ctx.view(torch.int16).clone()))
    return out


def _check(wl, sh, cf, tmp_path, name):
    dev = torch.device("cuda:0")
    W = weights_dev(wl)
    xs = [dev_tensor(wl, s) for s in wl.steps[:N_STEPS]]
    ctx = dev_tensor(wl, wl.ctx) if wl.n_ctx else None
    # uninterrupted chain
    ref = _run(wl, sh, cf, W, xs, ctx, oc.LayerCache(sh, dev), oc.workspace(sh, cf, dev), range(N_STEPS))
    # stopped after STOP_AFTER steps, checkpointed to a file
    cache = oc.LayerCache(sh, dev)
    first = _run(wl, sh, cf, W, xs, ctx, cache, oc.workspace(sh, cf, dev), range(STOP_AFTER))
    path = tmp_path / f"{name}.pt"
    torch.save({"y": cache.y.cpu(), "valid": cache.valid, "step": cache.step}, path)
    del cache
    torch.cuda.empty_cache()
    # resumed from the file into a fresh cache and workspace
    st = torch.load(path, weights_only=True)
    resumed = oc.LayerCache(sh, dev)
    resumed.y.copy_(st["y"].to(dev))
    resumed.valid, resumed.step = st["valid"], st["step"]
    assert resumed.valid == 1 and resumed.step == STOP_AFTER
    rest = _run(wl, sh, cf, W, xs, ctx, resumed, oc.workspace(sh, cf, dev), range(STOP_AFTER, N_STEPS))
    for s, (y, y_ctx) in enumerate(first + rest):
        assert torch.equal(y, ref[s][0]), f"{name}: step {s} output differs"
        if y_ctx is not None:
            assert torch.equal(y_ctx, ref[s][1]), f"{name}: step {s} context output differs"
    assert resumed.step == N_STEPS
    _say(f"{name}: steps {STOP_AFTER}..{N_STEPS - 1} resumed from the file match the uninterrupted chain")


@pytest.mark.parametrize("kw", [
    dict(gran="token", F=1, H=16, W=16, C=128, heads=2, head_dim=64, dtype="bf16", n_ctx=5),
    dict(gran="frame", F=6, H=8, W=8, C=64, heads=2, head_dim=32, dtype="bf16", r_frame=0.5),
    dict(gran="frame", F=8, H=8, W=8, C=64, heads=2, head_dim=32, dtype="bf16", r_frame=0.25, patch_k=2),
    dict(gran="block", F=9, H=8, W=8, C=128, heads=2, head_dim=64, dtype="bf16"),
    dict(gran="frame_token", F=7, H=8, W=8, C=64, heads=2, head_dim=32, dtype="bf16", r_frame=0.3),
    dict(gran="token", F=1, H=16, W=16, C=64, heads=2, head_dim=32, dtype="f32"),
], ids=["token_ctx", "frame", "frame_patches_k2", "block", "frame_token", "token_f32"])
def test_resume_small(kw, tmp_path):
    kw = dict(kw)
    gran = kw.pop("gran")
    wl = small_workload(gran, n_steps=N_STEPS, seed=21, **kw)
    sh, cf, _, _ = shapes(wl)
    _say(f"resume {gran} {kw}")
    _check(wl, sh, cf, tmp_path, gran)


def test_resume_sd3_layer(tmp_path):
    """The benchmarked layer: 4096 image + 333 text tokens, C = 1536, Token
    Cache r = 0.5."""
    wl = make_workload("sd3_1024", N_STEPS)
    sh, cf, _, _ = shapes(wl)
    _say("resume sd3_1024")
    _check(wl, sh, cf, tmp_path, "sd3_1024")
