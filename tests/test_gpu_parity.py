"""GPU parity of the HIP library against the CPU oracle (run on an MI355X).

Every test calls through the C ABI (via the thin Python binding) on seeded
synthetic inputs and compares with the oracle under the rules in
tests/parity.py.  Sizes span several tiles with ragged tails; the full-size
workloads run the launch configuration the benchmark times.
"""
import sys

import numpy as np
import pytest
import torch

from oc_synth import make_workload, small_workload
from oracle import oc_oracle as O
import paper_2607_23844_amd as oc

from parity import (TOL, RAW_TOL, check_output_bars, dev_tensor, layer_step_parity, layer_step_sampled_parity,
                    rel_err, shapes, to_f64, weights_dev, weights_f64, check_match, group_margins)

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    oc.lib()
    return torch.device("cuda:0")


def chain(wl, n_steps, cold="matched", gran=None, r=None, r_frame=None, patch_k=None, case="", coarse_k=0,
          r_coarse=0.0):
    sh, cf, osh, ocf = shapes(wl, gran, r, r_frame, patch_k, cold, coarse_k, r_coarse)
    dev = torch.device("cuda:0")
    ws = oc.workspace(sh, cf, dev)
    cache = oc.LayerCache(sh, dev)
    ctx_dev = dev_tensor(wl, wl.ctx) if wl.n_ctx else None
    ctx64 = wl.f64(wl.ctx) if wl.n_ctx else None
    W, W64 = weights_dev(wl), weights_f64(wl)
    ora, valid = None, False
    stats = []
    for s in range(n_steps):
        _say(f"  step {s} of {wl.name} gran={cf.gran} r={cf.r} rf={cf.r_frame} k={cf.patch_k} cold={cold}"
             + (f" coarse k={cf.coarse_k} r={cf.r_coarse}" if cf.coarse_k else ""))
        res, st = layer_step_parity(wl, wl.steps[s], sh, cf, osh, ocf, cache, ws, ora, valid, ctx_dev, ctx64, W, W64,
                                    case=case)
        _say(f"    {st}")
        stats.append(st)
        ora, valid = res.y, True
        assert cache.valid == 1 and cache.step == s + 1
    return stats


# ---------------------------------------------------------------------------
# small layers: every granularity, both dtypes, patches, context, head dims
# ---------------------------------------------------------------------------
SMALL = [
    dict(gran="token", F=1, H=8, W=8, C=32, heads=2, head_dim=16, dtype="f32"),
    dict(gran="token", F=2, H=8, W=8, C=32, heads=2, head_dim=16, dtype="f32", patch_k=2),
    dict(gran="token", F=1, H=16, W=16, C=64, heads=2, head_dim=32, dtype="bf16"),
    dict(gran="token", F=1, H=16, W=16, C=64, heads=2, head_dim=32, dtype="bf16", patch_k=2),
    dict(gran="token", F=1, H=12, W=20, C=64, heads=2, head_dim=32, dtype="bf16", n_ctx=7),
    dict(gran="token", F=3, H=16, W=12, C=144, heads=2, head_dim=72, dtype="bf16"),
    dict(gran="token", F=1, H=24, W=24, C=128, heads=2, head_dim=64, dtype="bf16", r=0.75, patch_k=3),
    dict(gran="block", F=6, H=8, W=8, C=64, heads=2, head_dim=16, dtype="bf16"),
    dict(gran="block", F=5, H=8, W=12, C=48, heads=3, head_dim=16, dtype="f32", patch_k=2),
    dict(gran="block", F=9, H=8, W=8, C=128, heads=2, head_dim=64, dtype="bf16"),
    dict(gran="frame", F=8, H=8, W=8, C=64, heads=2, head_dim=32, dtype="bf16", planted=True, r_frame=0.25),
    dict(gran="frame", F=7, H=4, W=8, C=32, heads=2, head_dim=16, dtype="f32", planted=True, r_frame=0.45),
    dict(gran="frame_token", F=7, H=8, W=8, C=64, heads=2, head_dim=32, dtype="bf16", r_frame=0.3, planted=True),
    dict(gran="frame_token", F=9, H=8, W=8, C=64, heads=2, head_dim=32, dtype="bf16", r_frame=0.45, patch_k=2,
         planted=True),
    dict(gran="frame_token", F=6, H=8, W=8, C=32, heads=2, head_dim=16, dtype="f32", r_frame=0.35, planted=True),
    # every candidate cached (r < 1 is required; floor(0.99 * 64) = 63 is
    # clamped to the 48 candidates): only the representatives (and the
    # context) are computed
    dict(gran="token", F=1, H=8, W=8, C=64, heads=2, head_dim=32, dtype="bf16", r=0.99, n_ctx=3),
    dict(gran="block", F=4, H=8, W=8, C=64, heads=2, head_dim=32, dtype="bf16", r=0.99),
    # Block Cache over 4096 positions: 3072 candidates, selected and
    # compacted by the 1024-thread selection block
    dict(gran="block", F=2, H=64, W=64, C=64, heads=2, head_dim=32, dtype="bf16"),
    # Frame Cache at its largest frame count (32), compacted by the frame
    # stage's final block
    dict(gran="frame", F=32, H=4, W=4, C=64, heads=2, head_dim=32, dtype="bf16", planted=True, r_frame=0.4),
    # Frame Cache on k x k patches (§3.3): per-patch tile decisions, frames
    # of varying length; the last case caches every odd tile of every patch
    # (odd frames keep no token at all)
    dict(gran="frame", F=8, H=16, W=16, C=64, heads=2, head_dim=32, dtype="bf16", r_frame=0.3, patch_k=2,
         frame_drift=0.3),
    dict(gran="frame", F=6, H=8, W=12, C=32, heads=2, head_dim=16, dtype="f32", r_frame=0.34, patch_k=2,
         frame_drift=0.3),
    dict(gran="frame", F=9, H=16, W=16, C=64, heads=2, head_dim=64, dtype="bf16", r_frame=0.25, patch_k=4,
         frame_drift=0.3),
    dict(gran="frame", F=7, H=8, W=8, C=64, heads=2, head_dim=32, dtype="bf16", r_frame=0.45, patch_k=2,
         frame_drift=0.3),
    # degenerate grids: one 2x2 window (three candidates, one representative),
    # two frames (one candidate frame), and a bf16 channel count that is not a
    # multiple of 64 (register-staged tiles instead of the DMA engine)
    dict(gran="token", F=1, H=2, W=2, C=16, heads=1, head_dim=16, dtype="bf16", r=0.5),
    dict(gran="frame", F=2, H=4, W=4, C=32, heads=2, head_dim=16, dtype="bf16", r_frame=0.6, planted=True),
    dict(gran="token", F=1, H=8, W=12, C=40, heads=1, head_dim=16, dtype="bf16", n_ctx=2),
]


@pytest.mark.parametrize("case", range(len(SMALL)))
@pytest.mark.parametrize("cold", ["matched", "full"])
def test_small_layer_chain(case, cold):
    kw = dict(SMALL[case])
    kw.setdefault("r", 0.5)
    wl = small_workload(n_steps=3, seed=100 + case, **kw)
    _say(f"case {case}: {kw} cold={cold}")
    chain(wl, 3, cold=cold)


@pytest.mark.parametrize("scale", [10, 30])
@pytest.mark.parametrize("gran,head_dim,F", [("token", 64, 1), ("block", 72, 8)])
def test_heavy_tailed_activations_chain(gran, head_dim, F, scale):
    """Activations with three outlier channels scaled by 10 or 30 over the
    rest (heavy-tailed channels of transformer activations): both output
    bars still hold with fp16 attention intermediates.  The limit is the
    attention logits, not fp16's range: a logit carries a relative error of
    about 2^-11 from the fp16 q and k, so the bars hold while the largest
    |q.k|/sqrt(head_dim) stays below about 100 (82 at scale 30 here); at
    scale 50 and beyond (logits of 2e2-1e5) the error grows past the bars,
    which the library's header states as its supported range."""
    from oc_synth import bf16_bits
    wl = small_workload(gran, F=F, H=16, W=16, C=256, heads=4, head_dim=head_dim, dtype="bf16", r=0.5,
                        n_steps=2, seed=61)
    steps = []
    for st in wl.steps:
        x = wl.to_f32(st).copy()
        x[..., [3, 77, 200]] *= np.float32(scale)
        steps.append(bf16_bits(x))
    wl.steps = steps
    x64 = wl.f64(wl.steps[0]).reshape(-1, wl.C)
    q, k = x64 @ wl.f64(wl.wq).T, x64 @ wl.f64(wl.wk).T
    top = max(float(np.abs(q[:, h * head_dim:(h + 1) * head_dim] @ k[:, h * head_dim:(h + 1) * head_dim].T).max())
              for h in range(wl.heads)) / np.sqrt(head_dim)
    _say(f"heavy-tailed {gran} x{scale}: largest |logit| {top:.3g}")
    assert top < 100
    chain(wl, 2)


# ---------------------------------------------------------------------------
# individual entry points
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("dtype,dh,n_seq,L,n_ctx", [
    ("bf16", 64, 1, 2381 - 333, 333), ("bf16", 64, 3, 130, 0), ("bf16", 64, 2, 700, 0), ("bf16", 64, 2, 256, 0),
    # head dim 64, at most 64 keys: projection and attention fused per tile of
    # whole sequences (ragged last tile; 2, 3, 5 and 128 sequences per tile)
    ("bf16", 64, 7, 25, 0), ("bf16", 64, 5, 64, 0), ("bf16", 64, 4, 33, 0), ("bf16", 64, 130, 1, 0), ("bf16", 72, 5, 77, 0), ("bf16", 72, 7, 16, 0),
    ("bf16", 16, 2, 9, 0), ("bf16", 128, 1, 200, 5), ("f32", 64, 1, 128, 0), ("f32", 16, 3, 33, 0),
    # the other supported head dims, long and short sequences
    ("bf16", 32, 2, 1000, 0), ("bf16", 48, 3, 100, 0), ("bf16", 80, 2, 150, 0), ("bf16", 96, 2, 300, 0),
    ("bf16", 128, 3, 40, 0), ("bf16", 96, 1, 70, 3),
    # K/V staged by DMA into padded K rows (head dims not a multiple of 64), ragged last tiles
    ("bf16", 48, 2, 333, 0), ("bf16", 80, 1, 700, 0), ("bf16", 16, 2, 260, 0), ("bf16", 72, 1, 456, 4),
    # grids too large for eight-wave blocks: four-wave register staging for wide heads (O scaled in place,
    # V fragments per key block) and four-wave DMA for head dim 128 (K fragments read per tile)
    ("bf16", 72, 90, 200, 0), ("bf16", 96, 90, 130, 0), ("bf16", 128, 86, 256, 0),
])
def test_attn_reduced_vs_oracle(dtype, dh, n_seq, L, n_ctx):
    _say(f"attn_reduced {dtype} dh={dh} n_seq={n_seq} L={L} n_ctx={n_ctx}")
    heads = 3 if dh != 64 or n_ctx == 0 else 24
    C = 256 if heads == 3 else 1536
    wl = small_workload("token", F=1, H=4, W=4, C=C, heads=heads, head_dim=dh, dtype=dtype, seed=5)
    rng = np.random.default_rng(3)
    sh = oc.Shape(1, 4, 4, C, heads, dh, n_ctx, dtype)
    xk = rng.standard_normal((n_seq, L, C)).astype(np.float32)
    ctx = rng.standard_normal((n_ctx, C)).astype(np.float32) if n_ctx else None
    from oc_synth import bf16_bits
    store = (lambda a: bf16_bits(a)) if dtype == "bf16" else (lambda a: a)
    xk_s = store(xk)
    ctx_s = store(ctx) if n_ctx else None
    y, yc = oc.attn_reduced(dev_tensor(wl, xk_s), n_seq, L, weights_dev(wl), sh,
                            ctx=dev_tensor(wl, ctx_s) if n_ctx else None)
    torch.cuda.synchronize()
    yk64, yc64 = O.attn_reduced(wl.f64(xk_s), wl.f64(ctx_s) if n_ctx else None, weights_f64(wl), heads, dh)
    e, raw = rel_err(to_f64(y), yk64, dtype), rel_err(to_f64(y), yk64)
    if n_ctx:
        e, raw = max(e, rel_err(to_f64(yc), yc64, dtype)), max(raw, rel_err(to_f64(yc), yc64))
    _say(f"  err {e:.3g} (raw {raw:.3g})")
    check_output_bars(e, raw, dtype, "attention output", case=f"attn {dtype} dh{dh} {n_seq}x{L}+{n_ctx}")


def test_gather_restore_bit_exact():
    wl = small_workload("token", F=2, H=8, W=8, C=64, heads=2, head_dim=32, dtype="bf16", seed=9)
    sh, cf, osh, ocf = shapes(wl, r=0.5)
    x = dev_tensor(wl, wl.steps[0])
    ws = oc.workspace(sh, cf, x.device)
    nm, ni = oc.match(x, sh, cf, ws)
    kept, cached, rmap = oc.select(nm, ni, sh, cf, ws)
    xk = oc.gather(x, kept, sh, cf)
    torch.cuda.synchronize()
    xs = x.view(torch.int16).cpu().numpy().reshape(-1, sh.C)
    k = kept.cpu().numpy()
    np.testing.assert_array_equal(xk.view(torch.int16).cpu().numpy().reshape(-1, sh.C), xs[k])
    # restore: kept rows from y_kept, -1 rows from the cache, in and out of place
    yk = torch.randn((len(k), sh.C), device=x.device).to(torch.bfloat16)
    cache = torch.randn((sh.F, sh.N, sh.C), device=x.device).to(torch.bfloat16)
    y = oc.restore(yk, rmap, sh, cache_y=cache)
    torch.cuda.synchronize()
    m = rmap.cpu().numpy()
    ref = cache.view(torch.int16).cpu().numpy().reshape(-1, sh.C).copy()
    ykn = yk.view(torch.int16).cpu().numpy()
    ref[m >= 0] = ykn[m[m >= 0]]
    np.testing.assert_array_equal(y.view(torch.int16).cpu().numpy().reshape(-1, sh.C), ref)
    c2 = cache.clone()
    oc.restore(yk, rmap, sh, cache_y=c2, y=c2)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(c2.view(torch.int16).cpu().numpy().reshape(-1, sh.C), ref)


@pytest.mark.parametrize("dtype,F,H,W,C", [
    ("bf16", 1, 64, 64, 1536),   # 48 units of 4 chunks per row: 16 positions per block
    ("bf16", 3, 37, 61, 320),    # 10 units per row: 64 positions per block, ragged last block
    ("bf16", 2, 13, 11, 24),     # rows of 3 chunks, one chunk per unit: 256 positions per block
    ("f32", 1, 9, 9, 40),        # 10 one-chunk units per row, a single partial block
    ("f32", 2, 16, 16, 64),      # 4 units of 4 chunks per row
])
def test_restore_in_place_bit_exact(dtype, F, H, W, C):
    """In-place restoration (cached positions keep their values) moves only
    the positions whose map names a row of y_kept; every other map value
    (-1, -2, negative, at or past n_rows) leaves the position untouched, with
    the cache as the output and with no cache at all."""
    rng = np.random.default_rng(F * 1000 + C)
    n_pos = F * H * W
    n_rows = max(1, int(0.4 * n_pos))
    sh = oc.Shape(F, H, W, C, 1, 16, 0, dtype)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    m = rng.integers(-3, n_rows + 3, size=n_pos).astype(np.int32)
    rmap = torch.from_numpy(m).cuda()
    yk = torch.randn((n_rows, C), device="cuda").to(tdt)
    base = torch.randn((F, H * W, C), device="cuda").to(tdt)
    iview = torch.int16 if dtype == "bf16" else torch.int32
    ref = base.view(iview).cpu().numpy().reshape(n_pos, C).copy()
    fresh = (m >= 0) & (m < n_rows)
    ref[fresh] = yk.view(iview).cpu().numpy()[m[fresh]]
    for with_cache in (True, False):
        y = base.clone()
        oc.restore(yk, rmap, sh, cache_y=y if with_cache else None, y=y)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(y.view(iview).cpu().numpy().reshape(n_pos, C), ref)


def test_select_is_exact_on_library_similarities():
    """The selection kernel is integer work: given the library's own fp32
    node_max, its cached set equals the definition (largest first, smallest id
    on ties) evaluated on exactly those values, with many deliberate ties."""
    wl = small_workload("token", F=1, H=32, W=32, C=64, heads=2, head_dim=32, dtype="bf16", seed=4)
    sh, cf, osh, ocf = shapes(wl, r=0.5, patch_k=2)
    x = dev_tensor(wl, wl.steps[0])
    ws = oc.workspace(sh, cf, x.device)
    nm, ni = oc.match(x, sh, cf, ws)
    # quantise the similarities to force many exact ties
    nmq = (torch.round(nm * 64) / 64).contiguous()
    nmq[torch.isinf(nm)] = -float("inf")
    kept, cached, rmap = oc.select(nmq, ni, sh, cf, ws)
    torch.cuda.synchronize()
    dec = O.decide(wl.f64(wl.steps[0]).reshape(osh.F, osh.N, osh.C), osh, ocf)
    v = nmq.cpu().numpy().astype(np.float64)
    expect = []
    for gi, g in enumerate(dec.groups):
        expect += O.select_cached(v[gi, :len(g.src)], g.src, g.R)
    np.testing.assert_array_equal(cached.cpu().numpy(), np.array(sorted(expect)))


@pytest.mark.parametrize("gran,F,k", [("token", 1, 1), ("block", 4, 1), ("frame", 4, 1), ("frame_token", 5, 1),
                                      ("frame", 4, 2)])
def test_r0_is_bit_identical_to_full_attention(gran, F, k):
    wl = small_workload(gran, F=F, H=16, W=16, C=64, heads=2, head_dim=32, dtype="bf16", seed=21)
    sh, cf, osh, ocf = shapes(wl, r=0.0, r_frame=0.0, patch_k=k)
    dev = torch.device("cuda:0")
    x = dev_tensor(wl, wl.steps[0])
    ws = oc.workspace(sh, cf, dev)
    cache = oc.LayerCache(sh, dev)
    y, _, _ = oc.layer_cached(x, weights_dev(wl), cache, sh, cf, ws=ws)
    yf, _ = oc.attn_full(x, weights_dev(wl), sh, cf, ws=ws)
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16), yf.view(torch.int16))


def test_repeat_runs_are_bit_identical():
    wl = small_workload("frame_token", F=7, H=8, W=8, C=64, heads=2, head_dim=32, dtype="bf16", r_frame=0.3, seed=2)
    sh, cf, osh, ocf = shapes(wl)
    dev = torch.device("cuda:0")
    x = dev_tensor(wl, wl.steps[0])
    ws = oc.workspace(sh, cf, dev)
    outs = []
    for _ in range(3):
        cache = oc.LayerCache(sh, dev)
        y, _, tr = oc.layer_cached(x, weights_dev(wl), cache, sh, cf, ws=ws, trace=True)
        torch.cuda.synchronize()
        outs.append((y.view(torch.int16).clone(), tr["restore_map"].clone(), tr["node_max"].clone()))
    for o in outs[1:]:
        assert all(torch.equal(a, b) for a, b in zip(o, outs[0]))


@pytest.mark.parametrize("kw", [
    dict(gran="token", F=1, H=16, W=16, C=128, heads=2, head_dim=64, dtype="bf16", n_ctx=5),
    dict(gran="block", F=9, H=8, W=8, C=128, heads=2, head_dim=64, dtype="bf16"),
    dict(gran="frame_token", F=7, H=8, W=8, C=64, heads=2, head_dim=32, dtype="bf16", r_frame=0.3, planted=True),
], ids=["token_ctx", "block_dh64", "frame_token"])
def test_graph_replay_matches_eager(kw):
    """A warm cached step captured once in a HIP graph and replayed, with the
    program's own eager work and synchronisations between the replays: every
    replay leaves the same layer output as the eager step (the step is
    idempotent on a warm cache: retained rows are rewritten, cached ones kept)."""
    from paper_2607_23844_amd.runner import LayerRunner
    kw = dict(kw)
    wl = small_workload(kw.pop("gran"), n_steps=2, seed=7, **kw)
    sh, cf, _, _ = shapes(wl)
    dev = torch.device("cuda:0")
    x0, x1 = dev_tensor(wl, wl.steps[0]), dev_tensor(wl, wl.steps[1])
    ctx = dev_tensor(wl, wl.ctx) if wl.n_ctx else None
    run = LayerRunner(sh, cf, weights_dev(wl), dev, ctx)
    run(x0)
    run(x1)
    torch.cuda.synchronize()
    ref = run.cache.y.view(torch.int16).clone()
    ref_ctx = run.y_ctx.view(torch.int16).clone() if ctx is not None else None
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run.use_current_stream()
        run(x1)
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run.use_current_stream()
        run(x1)
    run.use_current_stream()
    scratch = torch.zeros(1 << 20, device=dev)
    for i in range(4):
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(run.cache.y.view(torch.int16), ref), f"replay {i}"
        if ref_ctx is not None:
            assert torch.equal(run.y_ctx.view(torch.int16), ref_ctx), f"replay {i} (context rows)"
        scratch.add_(1.0)          # eager work between the replays
        torch.cuda.synchronize()
        run(x1)                    # and an eager step of the layer itself
        torch.cuda.synchronize()
        assert torch.equal(run.cache.y.view(torch.int16), ref), f"eager step after replay {i}"


# ---------------------------------------------------------------------------
# full-size workloads (the shapes the benchmark times)
# ---------------------------------------------------------------------------
def test_tok16_f32_chain():
    wl = make_workload("tok16_f32", 4)
    chain(wl, 4)


@pytest.mark.parametrize("k", [2, 4, 8])
def test_sd3_match_patch_sizes(k):
    wl = make_workload("sd3_1024", 1)
    sh, cf, osh, ocf = shapes(wl, r=0.5, patch_k=k)
    x = dev_tensor(wl, wl.steps[0])
    ws = oc.workspace(sh, cf, x.device)
    nm, ni = oc.match(x, sh, cf, ws)
    torch.cuda.synchronize()
    x64 = wl.f64(wl.steps[0])
    dec = O.decide(x64, osh, ocf)
    ov, worst = check_match(x64, dec, nm.cpu().numpy(), ni.cpu().numpy(), "token")
    _say(f"sd3 k={k}: node_max err {worst:.3g}, in-band idx differences {len(ov)}")


# two levels of the hierarchy (§3.3): patch-local first, then coarser
# patches or the whole frame among the candidates left
TWO_LEVEL = [
    (dict(gran="token", F=2, H=16, W=16, C=64, heads=2, head_dim=32, dtype="bf16"), 4, 0.25, 1, 0.25),
    (dict(gran="token", F=1, H=16, W=24, C=64, heads=2, head_dim=32, dtype="bf16", n_ctx=5), 4, 0.2, 2, 0.3),
    (dict(gran="token", F=1, H=16, W=16, C=32, heads=2, head_dim=16, dtype="f32"), 2, 0.3, 1, 0.2),
    (dict(gran="block", F=6, H=16, W=16, C=64, heads=2, head_dim=32, dtype="bf16"), 4, 0.25, 1, 0.25),
    (dict(gran="block", F=5, H=8, W=16, C=48, heads=3, head_dim=16, dtype="f32"), 2, 0.2, 1, 0.4),
    # the first level caches every candidate it may: the second finds none left
    (dict(gran="token", F=1, H=16, W=16, C=64, heads=2, head_dim=32, dtype="bf16"), 2, 0.9, 1, 0.5),
]


@pytest.mark.parametrize("case", range(len(TWO_LEVEL)))
@pytest.mark.parametrize("cold", ["matched", "full"])
def test_two_level_chain(case, cold):
    kw, k1, r1, k2, r2 = TWO_LEVEL[case]
    kw = dict(kw)
    wl = small_workload(n_steps=3, seed=300 + case, **kw)
    _say(f"two levels {case}: {kw} k={k1} r={r1} then k={k2} r={r2} cold={cold}")
    chain(wl, 3, cold=cold, r=r1, patch_k=k1, coarse_k=k2, r_coarse=r2)


@pytest.mark.parametrize("k1,r1,k2,r2", [(4, 0.25, 1, 0.25), (8, 0.3, 2, 0.2)])
def test_sd3_two_level_chain(k1, r1, k2, r2):
    """The SD3-like layer (4096 image + 333 text tokens): patch-local Token
    Cache, then a coarser level, cold and warm."""
    wl = make_workload("sd3_1024", 3)
    chain(wl, 3, r=r1, patch_k=k1, coarse_k=k2, r_coarse=r2)


@pytest.mark.parametrize("r", [0.25, 0.5, 0.75])
def test_sd3_chain(r):
    wl = make_workload("sd3_1024", 4 if r == 0.5 else 2)
    chain(wl, 4 if r == 0.5 else 2, r=r)


def test_latte_spatial_planted_chain():
    wl = make_workload("latte_spatial_planted", 3)
    chain(wl, 3)


def test_latte_spatial_chain():
    """The unplanted Latte-like spatial layer the benchmark times: its eight
    candidate frames' best similarities lie within 1e-4 of each other, so the
    frame decisions are in the band and the oracle takes the library's
    choices; the maps and outputs are then checked in full."""
    wl = make_workload("latte_spatial", 3)
    chain(wl, 3)


@pytest.mark.parametrize("k", [2, 4])
def test_latte_spatial_frame_patches_chain(k):
    """The Latte-like spatial layer with Frame Cache on k x k patches (§3.3):
    per-patch tile decisions and frames of varying length, three steps in
    full.  Frames that keep one or two patches have outputs far above the
    layer's RMS, so the raw bar is the one listed for these chains."""
    wl = make_workload("latte_spatial", 3)
    chain(wl, 3, patch_k=k, case=f"latte_spatial frame patches k{k}")


def test_latte_temporal_chain():
    wl = make_workload("latte_temporal", 2)
    chain(wl, 2)


# ---------------------------------------------------------------------------
# SVD-XT-like U-Net level at full size (25 frames of 72x128 tokens, C=320):
# decisions and maps in full, outputs on a seeded sample of positions
# ---------------------------------------------------------------------------
def sampled_chain(wl, n_steps, n_sample=256, seed=11):
    sh, cf, osh, ocf = shapes(wl)
    dev = torch.device("cuda:0")
    ws = oc.workspace(sh, cf, dev)
    cache = oc.LayerCache(sh, dev)
    W, W64 = weights_dev(wl), weights_f64(wl)
    rng = np.random.default_rng(seed)
    positions = np.sort(rng.choice(osh.F * osh.N, n_sample, replace=False))
    y_prev, valid, stats = None, False, []
    for s in range(n_steps):
        _say(f"  step {s} of {wl.name} gran={cf.gran} r={cf.r} rf={cf.r_frame} k={cf.patch_k} (sampled outputs)")
        y_prev, st = layer_step_sampled_parity(wl, wl.steps[s], sh, cf, osh, ocf, cache, ws, valid, W, W64,
                                               positions, y_prev)
        _say(f"    {st}")
        stats.append(st)
        valid = True
    return stats


@pytest.mark.parametrize("name", ["svdxt_level_planted", "svdxt_level", "svdxt_level_k4"])
def test_svdxt_level_spatial_sampled(name):
    wl = make_workload(name, 2)
    sampled_chain(wl, 2)


def test_svdxt_level_temporal_full_sampled():
    """The level's uncached temporal layer (its own weights): 9216 sequences
    of 25 frames, checked at a seeded sample of positions."""
    wl = make_workload("svdxt_level", 2)
    tw = wl.t_weights
    sh = oc.Shape(wl.F, wl.H, wl.W, wl.C, wl.heads, wl.head_dim, 0, wl.dtype)
    cf = oc.Cfg("block", 0.0, 0.0, 1, "matched")
    x = dev_tensor(wl, wl.steps[1])
    y, _ = oc.attn_full(x, weights_dev(wl, tw), sh, cf)
    torch.cuda.synchronize()
    x64 = wl.f64(wl.steps[1]).reshape(wl.F, wl.H * wl.W, wl.C)
    W64 = weights_f64(wl, tw)
    rng = np.random.default_rng(12)
    ns = np.sort(rng.choice(wl.H * wl.W, 96, replace=False))
    got = to_f64(y).reshape(wl.F, wl.H * wl.W, wl.C)[:, ns, :]
    ref = np.stack([O.multi_head_attention(x64[:, n, :], W64["wq"], W64["wk"], W64["wv"], W64["wo"], wl.heads,
                                           wl.head_dim) for n in ns], axis=1)
    err, raw = rel_err(got, ref, wl.dtype), rel_err(got, ref)
    _say(f"  temporal layer sampled error {err:.3g} (raw {raw:.3g})")
    check_output_bars(err, raw, wl.dtype, "temporal layer output")
