"""Pins of the oracle's two-level hierarchy (OmniCache §3.3: matching and
reuse first inside k x k patches, then in coarser patches or the whole
frame; reading R23).  The second level is checked against what does not
depend on the oracle itself: brute force over tiny grids with exact
rational sums, the two ways it reduces to a single level, and the static
counts that the library's plan relies on."""
import math

import numpy as np
import pytest

from oracle import brute as B
from oracle import oc_oracle as O


def _x(F, H, W, C, seed):
    return np.random.default_rng(seed).standard_normal((F, H * W, C))


def _brute_cascade(x, shape, cfg):
    """Both levels from scratch: per group, brute-force best matches against
    the group's representatives (descriptors: token rows, or the F rows of a
    block), then the exact optimum R-subset of the remaining candidates."""
    F, N, C = x.shape
    W = shape.W

    if cfg.gran == O.TOKEN:
        desc = {f * N + n: list(x[f, n]) for f in range(F) for n in range(N)}
    else:
        desc = {n: list(x[:, n, :].reshape(-1)) for n in range(N)}

    def groups(k):
        h, w = shape.H // k, shape.W // k
        frames = range(F) if cfg.gran == O.TOKEN else [None]
        out = []
        for f in frames:
            for py in range(k):
                for px in range(k):
                    items, dst, src = [], [], []
                    for y in range(py * h, (py + 1) * h):
                        for xx in range(px * w, (px + 1) * w):
                            i = (f * N if f is not None else 0) + y * W + xx
                            items.append(i)
                            (dst if y % 2 == 0 and xx % 2 == 0 else src).append(i)
                    out.append((items, dst, src))
        return out

    def level(k, ratio, exclude):
        cached, match = set(), {}
        for items, dst, src in groups(k):
            rest = [s for s in src if s not in exclude]
            R = min(int(math.floor(ratio * len(items) + 1e-9)), len(rest))
            bv, bi = B.brute_best_match(desc, rest, dst)
            sel = B.brute_select({s: bv[s] for s in rest}, R)
            cached |= set(sel)
            match.update({s: bi[s] for s in sel})
        return cached, match

    c1, m1 = level(cfg.patch_k, cfg.r, set())
    c2, m2 = level(cfg.coarse_k, cfg.r_coarse, c1)
    return c1, c2, {**m1, **m2}


def _oracle_levels(x, shape, cfg):
    dec = O.decide(x, shape, cfg)
    n1 = len(O.token_groups(shape, cfg.patch_k, range(shape.F), 0.0)) if cfg.gran == O.TOKEN else \
        len(O.block_groups(shape, cfg.patch_k, 0.0))
    c1 = set(i for c in dec.cached[:n1] for i in c)
    c2 = set(i for c in dec.cached[n1:] for i in c)
    match = {}
    for g, ni, c in zip(dec.groups, dec.node_idx, dec.cached):
        pos = {s: j for j, s in enumerate(g.src)}
        match.update({s: int(ni[pos[s]]) for s in c})
    return dec, c1, c2, match


@pytest.mark.parametrize("seed", [1, 2, 3])
@pytest.mark.parametrize("k1,k2,r1,r2", [(2, 1, 0.125, 0.0625), (4, 2, 0.25, 0.125), (4, 1, 0.125, 0.03125)])
def test_token_cascade_brute_force(seed, k1, k2, r1, r2):
    shape = O.LayerShape(1, 8, 8, 5, 1, 8)
    cfg = O.CacheCfg("token", r=r1, patch_k=k1, coarse_k=k2, r_coarse=r2)
    x = _x(1, 8, 8, 5, seed)
    _, c1, c2, match = _oracle_levels(x, shape, cfg)
    b1, b2, bm = _brute_cascade(x, shape, cfg)
    assert (c1, c2) == (b1, b2)
    assert match == bm


@pytest.mark.parametrize("seed", [4, 5])
def test_block_cascade_brute_force(seed):
    shape = O.LayerShape(3, 8, 8, 4, 1, 8)
    cfg = O.CacheCfg("block", r=0.125, patch_k=2, coarse_k=1, r_coarse=0.0625)
    x = _x(3, 8, 8, 4, seed)
    _, c1, c2, match = _oracle_levels(x, shape, cfg)
    b1, b2, bm = _brute_cascade(x, shape, cfg)
    assert (c1, c2) == (b1, b2)
    assert match == bm


@pytest.mark.parametrize("gran,F", [("token", 2), ("block", 4)])
def test_cascade_reduces_to_one_level(gran, F):
    """r_coarse = 0 is the first level alone; r = 0 leaves every candidate
    to the second level, which is then the single level at coarse_k."""
    shape = O.LayerShape(F, 16, 16, 8, 1, 8)
    x = _x(F, 16, 16, 8, 7)
    only1 = O.decide(x, shape, O.CacheCfg(gran, r=0.25, patch_k=4))
    casc0 = O.decide(x, shape, O.CacheCfg(gran, r=0.25, patch_k=4, coarse_k=2, r_coarse=0.0))
    assert set(i for c in casc0.cached for i in c) == set(i for c in only1.cached for i in c)
    only2 = O.decide(x, shape, O.CacheCfg(gran, r=0.3, patch_k=2))
    casc1 = O.decide(x, shape, O.CacheCfg(gran, r=0.0, patch_k=4, coarse_k=2, r_coarse=0.3))
    assert set(i for c in casc1.cached for i in c) == set(i for c in only2.cached for i in c)


@pytest.mark.parametrize("k1,k2,r1,r2", [(4, 1, 0.25, 0.25), (4, 2, 0.2, 0.2), (8, 2, 0.3, 0.4), (2, 1, 0.7, 0.7)])
def test_cascade_counts_are_static(k1, k2, r1, r2):
    """Every first-level patch caches its full budget, so a coarse patch
    always has (k1/k2)^2 * R1 fewer candidates: each frame keeps
    N - k1^2 R1 - k2^2 R2 tokens with R2 = min(floor(r2 n2), n2_src -
    (k1/k2)^2 R1) (the formula of the library's plan); the two levels are
    disjoint and no representative is cached."""
    F, H, W = 2, 16, 16
    shape = O.LayerShape(F, H, W, 8, 1, 8)
    cfg = O.CacheCfg("token", r=r1, patch_k=k1, coarse_k=k2, r_coarse=r2)
    dec, c1, c2, _ = _oracle_levels(_x(F, H, W, 8, 11), shape, cfg)
    n1 = (H // k1) * (W // k1)
    R1 = min(int(math.floor(r1 * n1 + 1e-9)), n1 - n1 // 4)
    n2 = (H // k2) * (W // k2)
    R2 = min(int(math.floor(r2 * n2 + 1e-9)), n2 - n2 // 4 - (k1 // k2) ** 2 * R1)
    assert not (c1 & c2)
    assert len(c1) == F * k1 * k1 * R1 and len(c2) == F * k2 * k2 * R2
    reps = {f * H * W + y * W + x for f in range(F) for y in range(0, H, 2) for x in range(0, W, 2)}
    assert not ((c1 | c2) & reps)
    seqs = O.build_sequences(shape, cfg, dec)
    assert [len(s) for s in seqs] == [H * W - k1 * k1 * R1 - k2 * k2 * R2] * F


def test_cascade_layer_step_matches_single_level_at_zero():
    """The whole layer call with r_coarse = 0 equals the single level."""
    F, H, W, C = 1, 16, 16, 16
    shape = O.LayerShape(F, H, W, C, 2, 8)
    rng = np.random.default_rng(3)
    x = rng.standard_normal((F, H * W, C))
    w = {k: rng.standard_normal((16, C)) / math.sqrt(C) for k in ("wq", "wk", "wv")}
    w["wo"] = rng.standard_normal((C, 16)) / 4.0
    a = O.layer_step(x, None, w, shape, O.CacheCfg("token", r=0.25, patch_k=4), None, False)
    b = O.layer_step(x, None, w, shape, O.CacheCfg("token", r=0.25, patch_k=4, coarse_k=1, r_coarse=0.0), None, False)
    np.testing.assert_array_equal(a.kept_idx, b.kept_idx)
    np.testing.assert_array_equal(a.restore_map, b.restore_map)
    np.testing.assert_array_equal(a.y, b.y)


def test_cascade_rejects_bad_scopes():
    shape = O.LayerShape(1, 16, 16, 8, 1, 8)
    x = _x(1, 16, 16, 8, 1)
    for cfg in (O.CacheCfg("token", r=0.2, patch_k=4, coarse_k=3, r_coarse=0.1),
                O.CacheCfg("token", r=0.2, patch_k=2, coarse_k=2, r_coarse=0.1),
                O.CacheCfg("frame", r_frame=0.2, patch_k=2, coarse_k=1, r_coarse=0.1)):
        with pytest.raises(ValueError):
            O.decide(x, shape, cfg)
