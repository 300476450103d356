"""GPU parity of the feed-forward sublayer under the attention's selection
(oc_ffn_reduced) against the CPU oracle's feed_forward / ffn_step (the SD3
experiments cache attention and FFN layers alike, OmniCache §4.2).  Small
ragged cases check both output modes and index handling element by
element; the SD3-sized layer runs a cold and a warm step under the
selection of the cached attention call of the same step."""
import sys

import numpy as np
import pytest
import torch

from oc_synth import bf16_bits, bf16_bits_to_f32, ffn_weights, make_workload
from oracle import oc_oracle as O
import paper_2607_23844_amd as oc

from parity import check_output_bars, dev_tensor, rel_err, shapes, to_f64, weights_dev

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    oc.lib()


def _bf(a):
    return torch.from_numpy(np.ascontiguousarray(bf16_bits(a)).view(np.int16)).view(torch.bfloat16).cuda()


def _f64(t):
    return to_f64(t)


@pytest.mark.parametrize("F,H,W,C,hidden,n_rows,idx_kind", [
    (1, 8, 8, 64, 256, 37, "perm"),          # ragged rows, one tile of each kind
    (2, 16, 16, 128, 512, 300, "perm"),      # several row and hidden tiles, ragged
    (1, 16, 16, 192, 384, 256, "none"),      # identity rows, C not a power of two
    (3, 8, 8, 64, 64 * 13, 129, "perm"),     # hidden 832: 192-wide tiles with a ragged last one
    (1, 8, 8, 64, 256, 1, "perm"),           # a single row
])
@pytest.mark.parametrize("scatter", [True, False])
def test_ffn_small_vs_oracle(F, H, W, C, hidden, n_rows, idx_kind, scatter):
    _say(f"ffn F={F} {H}x{W} C={C} hidden={hidden} rows={n_rows} idx={idx_kind} scatter={scatter}")
    rng = np.random.default_rng(C + hidden + n_rows)
    FN = F * H * W
    x32 = rng.standard_normal((F, H * W, C)).astype(np.float32)
    w = ffn_weights(C, hidden, "bf16", seed=hidden)
    sh = oc.Shape(F, H, W, C, 1, 64, 0, "bf16")
    idx = np.sort(rng.choice(FN, n_rows, replace=False)).astype(np.int32) if idx_kind == "perm" else None
    if idx is not None:
        idx = rng.permutation(idx).astype(np.int32)       # any order
    x = _bf(x32)
    Wt = {k: torch.from_numpy(v.view(np.int16)).view(torch.bfloat16).cuda() for k, v in w.items()}
    y0 = torch.randn((F, H * W, C), device="cuda").to(torch.bfloat16) if scatter else None
    prev = y0.clone() if scatter else None
    kept = torch.from_numpy(idx).cuda() if idx is not None else None
    y = oc.ffn_reduced(x, Wt, sh, kept_idx=kept, n_rows=n_rows, y=y0, scatter=scatter)
    torch.cuda.synchronize()
    x64 = bf16_bits_to_f32(bf16_bits(x32)).astype(np.float64).reshape(FN, C)
    w1 = bf16_bits_to_f32(w["w1"]).astype(np.float64)
    w2 = bf16_bits_to_f32(w["w2"]).astype(np.float64)
    rows = idx if idx is not None else np.arange(n_rows)
    ref = O.feed_forward(x64[rows], w1, w2)
    if scatter:
        got = _f64(y).reshape(FN, C)
        untouched = np.setdiff1d(np.arange(FN), rows)
        assert torch.equal(y.view(torch.int16).reshape(FN, C)[torch.from_numpy(untouched).cuda()],
                           prev.view(torch.int16).reshape(FN, C)[torch.from_numpy(untouched).cuda()])
        got = got[rows]
    else:
        got = _f64(y)
    err, raw = rel_err(got, ref, "bf16"), rel_err(got, ref)
    _say(f"  error {err:.3g} (raw {raw:.3g})")
    check_output_bars(err, raw, "bf16", "feed-forward output")


def test_ffn_indices_outside_the_tensor_are_skipped():
    """Entries of kept_idx outside [0, F*N) are not read, and their rows of
    y are not written, in either output mode."""
    F, H, W, C, hidden = 1, 8, 8, 64, 256
    FN = F * H * W
    rng = np.random.default_rng(9)
    x = _bf(rng.standard_normal((F, H * W, C)).astype(np.float32))
    w = ffn_weights(C, hidden, "bf16", seed=1)
    Wt = {k: torch.from_numpy(v.view(np.int16)).view(torch.bfloat16).cuda() for k, v in w.items()}
    sh = oc.Shape(F, H, W, C, 1, 64, 0, "bf16")
    idx = torch.tensor([3, -1, 7, FN, 11, 1 << 30], dtype=torch.int32, device="cuda")
    y0 = torch.zeros((F, H * W, C), device="cuda", dtype=torch.bfloat16)
    y = oc.ffn_reduced(x, Wt, sh, kept_idx=idx, y=y0.clone(), scatter=True)
    ref = oc.ffn_reduced(x, Wt, sh, kept_idx=torch.tensor([3, 7, 11], dtype=torch.int32, device="cuda"),
                         y=y0.clone(), scatter=True)
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16), ref.view(torch.int16))
    sentinel = torch.full((6, C), 7.0, device="cuda", dtype=torch.bfloat16)
    yc = oc.ffn_reduced(x, Wt, sh, kept_idx=idx, y=sentinel.clone(), scatter=False)
    torch.cuda.synchronize()
    for r in (1, 3, 5):
        assert torch.equal(yc[r], sentinel[r])
    for r, t in ((0, 3), (2, 7), (4, 11)):
        assert torch.equal(yc[r].view(torch.int16), y.reshape(FN, C)[t].view(torch.int16))


def test_ffn_sd3_chain_under_the_attention_selection():
    """SD3-sized layer (4096 image tokens, C=1536, hidden 6144): step 0 is
    cold ("matched": the retained rows into a compact buffer, then oc_restore
    with the attention call's cold restore map), step 1 warm (the retained
    rows written in place into the FFN cache, cached rows left as they
    were).  Decisions come from oc_layer_cached's trace of the same step;
    outputs are compared with the oracle at 512 sampled positions, kept and
    cached alike."""
    wl = make_workload("sd3_1024", 2)
    sh, cf, osh, ocf = shapes(wl)
    dev = torch.device("cuda:0")
    hidden = 4 * wl.C
    w = ffn_weights(wl.C, hidden, "bf16")
    Wf = {k: torch.from_numpy(v.view(np.int16)).view(torch.bfloat16).cuda() for k, v in w.items()}
    w1 = wl.f64(w["w1"])
    w2 = wl.f64(w["w2"])
    Wa = weights_dev(wl)
    ctx = dev_tensor(wl, wl.ctx)
    ws = oc.workspace(sh, cf, dev)
    cache = oc.LayerCache(sh, dev)
    ffn_cache = torch.empty((wl.F, wl.N, wl.C), dtype=torch.bfloat16, device=dev)
    rng = np.random.default_rng(17)
    FN = wl.F * wl.N
    pos = np.sort(rng.choice(FN, 512, replace=False))
    prev_ref, prev_gpu = None, None
    for s in range(2):
        x = dev_tensor(wl, wl.steps[s])
        _, _, tr = oc.layer_cached(x, Wa, cache, sh, cf, ctx=ctx, ws=ws, trace=True)
        kept, rmap = tr["kept_idx"], tr["restore_map"]
        if s == 0:
            yk = oc.ffn_reduced(x, Wf, sh, kept_idx=kept, scatter=False)
            oc.restore(yk, rmap, sh, cache_y=None, y=ffn_cache)
        else:
            oc.ffn_reduced(x, Wf, sh, kept_idx=kept, y=ffn_cache, scatter=True)
        torch.cuda.synchronize()
        k_np, m_np = kept.cpu().numpy(), rmap.cpu().numpy()
        x64 = wl.f64(wl.steps[s]).reshape(FN, wl.C)
        # the oracle's chain at the sampled positions: a position reads the
        # fresh FFN output of the retained token its map names, or keeps the
        # previous step's value (restore map -1)
        src = np.array([k_np[m_np[p]] if m_np[p] >= 0 else -1 for p in pos])
        fresh = src >= 0
        ref = np.empty((len(pos), wl.C))
        ref[fresh] = O.feed_forward(x64[src[fresh]], w1, w2)
        if not fresh.all():
            assert prev_ref is not None, "a position restored from an empty cache"
            ref[~fresh] = prev_ref[~fresh]
        got_all = _f64(ffn_cache).reshape(FN, wl.C)
        got = got_all[pos]
        err, raw = rel_err(got, ref, "bf16"), rel_err(got, ref)
        _say(f"  step {s}: {int(fresh.sum())} fresh / {len(pos)} sampled, error {err:.3g} (raw {raw:.3g})")
        check_output_bars(err, raw, "bf16", "feed-forward output")
        if prev_gpu is not None:
            # cached positions keep the previous step's values bit for bit
            cached = np.nonzero(m_np < 0)[0]
            assert len(cached) == FN - len(k_np) and np.array_equal(got_all[cached], prev_gpu[cached])
        prev_ref, prev_gpu = ref, got_all
