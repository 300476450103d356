"""Helpers that compare the HIP library with the CPU oracle.

Decision parity (OmniCache §3.2 matching and selection):
  * node_idx must equal the oracle's wherever the oracle's top-two similarity
    margin exceeds BAND;
  * a candidate whose oracle best-match similarity is more than BAND away
    from its group's threshold (the R-th largest) must be cached on both
    sides or on neither; counts are always exact;
  * kept_idx and restore_map must equal, bit for bit, those of the oracle
    run with the library's in-band choices forced on it;
  * outputs, two bars, both asserted on every checked element:
      raw:      max |y - y_oracle| / RMS(y_oracle) <= 2e-2 (bf16) or 1e-4 (fp32);
      adjusted: max (|y - y_oracle| - u(y_oracle)) / RMS(y_oracle) <= 1e-2 (bf16),
                u(v) = half a bf16 ulp of v, the part of the difference that
                rounding the exact result to a bf16 output accounts for.
    Half a bf16 ulp is 2^-9 to 2^-8 of |v|, so the adjusted bar is the
    tighter one wherever |y_oracle| is below about 2.5-5 times the RMS; the
    raw bar caps the error at the peaks, where half an ulp is itself a
    large fraction of the RMS.
"""
from __future__ import annotations

import numpy as np
import torch

from oracle import oc_oracle as O
import paper_2607_23844_amd as oc

BAND = 1e-4
TOL = {"bf16": 1e-2, "f32": 1e-4}        # rounding-adjusted bar (rel_err with out_dtype)
RAW_TOL = {"bf16": 2e-2, "f32": 1e-4}    # raw bar: max |y - y_oracle| / RMS(y_oracle)
NODE_MAX_TOL = {"token": 2e-6, "block": 2e-6, "frame": 1e-5}


def dev_tensor(wl, arr) -> torch.Tensor:
    if wl.dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(arr)).cuda()


def weights_dev(wl, w=None):
    w = w or dict(wq=wl.wq, wk=wl.wk, wv=wl.wv, wo=wl.wo)
    return {k: dev_tensor(wl, v) for k, v in w.items()}


def weights_f64(wl, w=None):
    w = w or dict(wq=wl.wq, wk=wl.wk, wv=wl.wv, wo=wl.wo)
    return {k: wl.f64(v) for k, v in w.items()}


def to_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def shapes(wl, gran=None, r=None, r_frame=None, patch_k=None, cold="matched", coarse_k=0, r_coarse=0.0):
    gran = gran or wl.gran
    r = wl.r if r is None else r
    r_frame = wl.r_frame if r_frame is None else r_frame
    k = wl.patch_k if patch_k is None else patch_k
    sh = oc.Shape(wl.F, wl.H, wl.W, wl.C, wl.heads, wl.head_dim, wl.n_ctx, wl.dtype)
    cf = oc.Cfg(gran, r, r_frame, k, cold, coarse_k, r_coarse)
    osh = O.LayerShape(wl.F, wl.H, wl.W, wl.C, wl.heads, wl.head_dim, wl.n_ctx)
    ocf = O.CacheCfg(gran, r, r_frame, k, cold, coarse_k, r_coarse)
    return sh, cf, osh, ocf


def rel_err(y: np.ndarray, ref: np.ndarray, out_dtype: str = "f32") -> float:
    """Largest |y - ref| over RMS(ref).  For bf16 outputs the part that the
    final rounding of ref to bf16 accounts for (half a bf16 ulp of ref, 8
    significant bits) is taken off every element first: a correctly rounded
    result scores 0, and what remains is the error of the computation
    itself."""
    rms = float(np.sqrt(np.mean(ref * ref)))
    d = np.abs(y - ref)
    if out_dtype == "bf16":
        _, e = np.frexp(np.abs(ref))          # |ref| = f * 2^e, f in [0.5, 1)
        d = np.maximum(d - np.ldexp(1.0, e - 9), 0.0)
    return float(np.max(d)) / max(rms, 1e-30)


# Cases whose raw error exceeds the raw bar although the rounding-adjusted
# error is far inside its own: the excess is the final rounding of a peak
# output to bf16 (half an ulp of a value 8.7 times the RMS is 1.7-3.4% of
# the RMS).  Each entry: measured raw error, and the bar used for it.
RAW_EXCEPTIONS = {
    # 2 sequences of 256 tokens, 3 heads of 64: peak/RMS 8.7; measured raw
    # 0.0204, rounding-adjusted 0.0020
    "attn bf16 dh64 2x256+0": (0.0204, 0.025),
    # Latte-like spatial layer, Frame Cache on 2x2 / 4x4 patches: frames that
    # keep one or two patches (16-128 tokens) give outputs up to 13.3 times
    # the layer's RMS, where half a bf16 ulp alone is 2.75% of the RMS;
    # measured raw 0.0283 (k = 2, third step) and 0.0280 (k = 4), adjusted
    # 0.0014-0.0018
    "latte_spatial frame patches k2": (0.0283, 0.035),
    "latte_spatial frame patches k4": (0.0280, 0.035),
    # 2 sequences of 1000 tokens, 3 heads of 32: the peak output (5.95 times
    # the RMS) lies just below a power of two, where half a bf16 ulp is
    # 0.0198 of the RMS; measured raw 0.0224, rounding-adjusted 0.0026
    "attn bf16 dh32 2x1000+0": (0.0224, 0.03),
}


def check_output_bars(err: float, raw: float, dtype: str, what: str = "output", case: str = "") -> None:
    """Both output bars: the rounding-adjusted one and the raw one (for a
    case listed in RAW_EXCEPTIONS, the raw bar stated there)."""
    assert err <= TOL[dtype], f"{what}: error {err:.3g} > {TOL[dtype]} (rounding-adjusted)"
    raw_bar = RAW_EXCEPTIONS[case][1] if case in RAW_EXCEPTIONS else RAW_TOL[dtype]
    assert raw <= raw_bar, f"{what}: raw error {raw:.3g} > {raw_bar}"


def group_margins(x64: np.ndarray, g: O.Group, shape=None, k: int = 1) -> np.ndarray:
    """Per candidate: top-1 minus top-2 cosine similarity (inf with one rep)."""
    if g.kind == "frame_patch":
        S = O.cosine_matrix(O.tile_descriptors(x64, shape, k, g.src), O.tile_descriptors(x64, shape, k, g.dst))
    else:
        S = O.cosine_matrix(O.descriptors(x64, g.kind, g.src), O.descriptors(x64, g.kind, g.dst))
    if S.shape[1] < 2:
        return np.full(S.shape[0], np.inf)
    top = np.sort(S, axis=1)
    return top[:, -1] - top[:, -2]


def check_match(x64, dec: O.Decisions, nm_gpu: np.ndarray, ni_gpu: np.ndarray, kind: str, shape=None, k: int = 1):
    """node_max within tolerance; node_idx equal outside the margin band.
    Returns {candidate id: gpu rep id} for in-band disagreements."""
    tol = NODE_MAX_TOL[kind]
    overrides = {}
    worst = 0.0
    for gi, g in enumerate(dec.groups):
        n = len(g.src)
        d = np.abs(nm_gpu[gi, :n].astype(np.float64) - dec.node_max[gi])
        worst = max(worst, float(d.max()) if n else 0.0)
        assert np.all(d <= tol), f"group {gi}: node_max off by {d.max():.3g} > {tol}"
        assert np.all(nm_gpu[gi, n:] == -np.inf) and np.all(ni_gpu[gi, n:] == -1)
        diff = np.nonzero(ni_gpu[gi, :n] != dec.node_idx[gi])[0]
        if len(diff):
            marg = group_margins(x64, g, shape, k)
            for i in diff:
                assert marg[i] <= BAND, f"group {gi} cand {g.src[i]}: idx {ni_gpu[gi, i]} vs {dec.node_idx[gi][i]}, " \
                                        f"margin {marg[i]:.3g}"
                overrides[int(g.src[i])] = int(ni_gpu[gi, i])
    return overrides, worst


def check_selection(dec: O.Decisions, gpu_cached_items: set):
    """Same cached/kept status outside the band around each group's threshold;
    exact counts.  Returns the number of in-band disagreements."""
    n_diff = 0
    for gi, g in enumerate(dec.groups):
        gset = set(i for i in g.src if i in gpu_cached_items)
        assert len(gset) == g.R, f"group {gi}: {len(gset)} cached, budget {g.R}"
        oset = set(dec.cached[gi])
        if gset == oset:
            continue
        vals = np.sort(dec.node_max[gi])[::-1]
        tau = vals[g.R - 1] if g.R > 0 else np.inf
        pos = {s: i for i, s in enumerate(g.src)}
        for item in gset ^ oset:
            v = dec.node_max[gi][pos[item]]
            assert abs(v - tau) <= BAND, f"group {gi} item {item}: similarity {v} vs threshold {tau}"
            n_diff += 1
    return n_diff


def gpu_cached_items(kind_gran: str, cached_idx: np.ndarray, N: int, shape=None, k: int = 1) -> set:
    if kind_gran == "block":
        return set(int(p) % N for p in cached_idx)
    if kind_gran == "frame" and k > 1:
        # Frame Cache on patches: the tiles (top-left token ids) of the cached tokens
        h, w = shape.H // k, shape.W // k
        out = set()
        for p in cached_idx:
            f, n = divmod(int(p), N)
            y, x = divmod(n, shape.W)
            out.add(f * N + (y // h) * h * shape.W + (x // w) * w)
        return out
    if kind_gran == "frame":
        return set(int(p) // N for p in cached_idx)
    return set(int(p) for p in cached_idx)


def check_frame_stage(x64, osh, ocf, dec: O.Decisions, fmax, fidx, pairs):
    """Frame similarities, frame selection and pairing (frame_token)."""
    fg = dec.frame_group
    d = np.abs(np.asarray(fmax, np.float64) - dec.frame_max)
    assert np.all(d <= NODE_MAX_TOL["frame"]), d.max()
    marg = group_margins(x64, fg)
    for i, (a, b) in enumerate(zip(fidx, dec.frame_idx)):
        assert a == b or marg[i] <= BAND
    g_order = [int(s) for s, _ in pairs]
    assert len(g_order) == fg.R
    gset, oset = set(g_order), set(dec.frame_cached_order)
    if gset != oset:
        vals = np.sort(dec.frame_max)[::-1]
        tau = vals[fg.R - 1]
        pos = {s: i for i, s in enumerate(fg.src)}
        for f in gset ^ oset:
            assert abs(dec.frame_max[pos[f]] - tau) <= BAND
    # pairing: each chosen rep frame is, among the free ones, within the band of the best
    S = dec.frame_sim
    spos = {s: i for i, s in enumerate(fg.src)}
    dpos = {dd: j for j, dd in enumerate(fg.dst)}
    taken = set()
    for s, dd in pairs:
        s, dd = int(s), int(dd)
        free = [j for j in fg.dst if j not in taken]
        best = max(S[spos[s], dpos[j]] for j in free)
        assert dd in free and S[spos[s], dpos[dd]] >= best - BAND
        taken.add(dd)
    return dict(frame_order=g_order, pairs=[(int(s), int(dd)) for s, dd in pairs])


def _part(dec: O.Decisions, lo: int, hi: int) -> O.Decisions:
    return O.Decisions(dec.groups[lo:hi], dec.node_max[lo:hi], dec.node_idx[lo:hi], dec.cached[lo:hi])


def decision_parity_two_levels(x64, osh, ocf, tr, valid):
    """The same for a two-level hierarchy (coarse_k > 0).  The trace holds the
    first level's similarities; the library's selection is exact on them, so
    its first-level cached set is the definition applied to those values.
    That set is checked against the oracle's first level (band rule), the
    oracle's second level is formed from it, and the rest of the library's
    cached tokens is checked against that second level.  On a cold "matched"
    step the restore map names the representative each cached token was
    matched with; the second level's are checked against the oracle's
    margins and forced where in band."""
    no_skip = (not valid) and ocf.cold == O.COLD_FULL
    kind = "block" if ocf.gran == O.BLOCK else "token"
    nm = tr["node_max"].cpu().numpy()
    ni = tr["node_idx"].cpu().numpy()
    n1 = nm.shape[0]
    dec0 = O.decide(x64, osh, ocf, no_skip=no_skip)
    ov, worst_nm = check_match(x64, _part(dec0, 0, n1), nm, ni, kind, osh, ocf.patch_k)
    first = set()
    for gi, g in enumerate(dec0.groups[:n1]):
        first |= set(O.select_cached(nm[gi, :len(g.src)].astype(np.float64), g.src, g.R))
    n_band = check_selection(_part(dec0, 0, n1), first)
    dec1 = O.decide(x64, osh, ocf, no_skip=no_skip, forced={"cached_first": first})
    items = gpu_cached_items(ocf.gran, tr["cached_idx"].cpu().numpy(), osh.N, osh, ocf.patch_k)
    assert first <= items
    n_band += check_selection(_part(dec1, n1, len(dec1.groups)), items - first)
    if not valid and ocf.cold == O.COLD_MATCHED and not no_skip:
        kept = tr["kept_idx"].cpu().numpy()
        rmap = tr["restore_map"].cpu().numpy()
        N = osh.N
        for gi in range(n1, len(dec1.groups)):
            g = dec1.groups[gi]
            pos = {s_: i for i, s_ in enumerate(g.src)}
            marg = None
            for item in items - first:
                if item not in pos:
                    continue
                # the token whose row this cached item was restored from
                tok = int(item) if kind == "token" else int(item)
                src_tok = int(kept[rmap[tok]])
                rep = src_tok if kind == "token" else src_tok % N
                want = int(dec1.node_idx[gi][pos[item]])
                if rep != want:
                    marg = group_margins(x64, g, osh, ocf.coarse_k) if marg is None else marg
                    assert marg[pos[item]] <= BAND, f"coarse group {gi} item {item}: rep {rep} vs {want}"
                    ov[int(item)] = rep
    forced = dict(cached_first=first, cached=items, match=ov)
    dec = O.decide(x64, osh, ocf, no_skip=no_skip, forced=forced)
    return dec, forced, dict(node_max_err=worst_nm, in_band=n_band, idx_overrides=len(ov))


def decision_parity(x64, osh, ocf, tr, valid):
    """Matching and selection of one oc_layer_cached call (its trace) against
    the oracle; returns the oracle's decisions with the library's in-band
    choices forced on them, the forcing, and statistics."""
    if ocf.coarse_k:
        return decision_parity_two_levels(x64, osh, ocf, tr, valid)
    no_skip = (not valid) and ocf.cold == O.COLD_FULL
    forced = {}
    dec = O.decide(x64, osh, ocf, no_skip=no_skip)
    if ocf.gran == O.FRAME_TOKEN and not no_skip:
        forced.update(check_frame_stage(x64, osh, ocf, dec, tr["frame_max"].cpu().numpy(),
                                        tr["frame_idx"].cpu().numpy(), tr["pairs"].cpu().numpy()))
        if forced["frame_order"] != list(dec.frame_cached_order) or \
                [tuple(p) for p in forced["pairs"]] != [tuple(p) for p in dec.pairs]:
            dec = O.decide(x64, osh, ocf, no_skip=no_skip, forced=dict(forced))
    kind = "block" if ocf.gran == O.BLOCK else ("frame" if ocf.gran == O.FRAME else "token")
    nm = tr["node_max"].cpu().numpy()
    ni = tr["node_idx"].cpu().numpy()
    ov, worst_nm = check_match(x64, dec, nm, ni, kind, osh, ocf.patch_k)
    cached_idx = tr["cached_idx"].cpu().numpy()
    items = gpu_cached_items(ocf.gran, cached_idx, osh.N, osh, ocf.patch_k)
    n_band = check_selection(dec, items)
    forced.update(cached=items, match=ov)
    dec = O.force_decisions(dec, items, ov)
    return dec, forced, dict(node_max_err=worst_nm, in_band=n_band, idx_overrides=len(ov))


def check_maps(tr, kept_idx, cached_idx, restore_map):
    np.testing.assert_array_equal(tr["kept_idx"].cpu().numpy(), kept_idx)
    np.testing.assert_array_equal(tr["cached_idx"].cpu().numpy(), cached_idx)
    np.testing.assert_array_equal(tr["restore_map"].cpu().numpy(), restore_map)


def check_layer_step(x64, ctx64, W64, osh, ocf, ora_cache, valid, y, y_ctx, tr, dtype, case=""):
    """Checks one finished layer call (its output y, context output and
    trace) against the oracle step on the exact input x64, with the
    library's in-band choices forced on the oracle.  Returns the oracle's
    StepResult and statistics."""
    x64 = np.asarray(x64, dtype=np.float64).reshape(osh.F, osh.N, osh.C)
    _, forced, st = decision_parity(x64, osh, ocf, tr, valid)
    res = O.layer_step(x64, ctx64, W64, osh, ocf, ora_cache, valid, forced=forced)
    check_maps(tr, res.kept_idx, res.cached_idx, res.restore_map)
    yg = to_f64(y).reshape(res.y.shape)
    err, raw = rel_err(yg, res.y, dtype), rel_err(yg, res.y)
    if ctx64 is not None:
        yc = to_f64(y_ctx)
        err, raw = max(err, rel_err(yc, res.y_ctx, dtype)), max(raw, rel_err(yc, res.y_ctx))
    check_output_bars(err, raw, dtype, "layer output", case)
    st.update(err=err, err_raw=raw)
    return res, st


def layer_step_parity(wl, x_np, sh, cf, osh, ocf, cache, ws, ora_cache, valid, ctx_dev=None, ctx64=None,
                      W=None, W64=None, case=""):
    """One oc_layer_cached step against the oracle (with in-band forcing).
    Returns the oracle's StepResult and the statistics."""
    W = W or weights_dev(wl)
    W64 = W64 or weights_f64(wl)
    x = dev_tensor(wl, x_np)
    y, y_ctx, tr = oc.layer_cached(x, W, cache, sh, cf, ctx=ctx_dev, ws=ws, trace=True)
    torch.cuda.synchronize()
    return check_layer_step(wl.f64(x_np), ctx64, W64, osh, ocf, ora_cache, valid, y, y_ctx, tr, wl.dtype, case)


def sampled_outputs(x64, W64, osh, seqs, kept_idx, restore_map, positions, y_prev):
    """Oracle layer outputs at the given positions only: a retained position
    (or, on a cold step, a cached one mapped to a retained row) is computed by
    attention restricted to that query over its whole sequence; a position
    restored from the cache takes y_prev (the previous step's values at the
    same positions)."""
    xf = x64.reshape(-1, osh.C)
    where = {}
    for qi, sq in enumerate(seqs):
        for j, p in enumerate(sq):
            where[p] = (qi, j)
    out = np.empty((len(positions), osh.C))
    need = {}
    for i, p in enumerate(positions):
        r = int(restore_map[p])
        if r >= 0:
            qi, j = where[int(kept_idx[r])]
            need.setdefault(qi, []).append((i, j))
        else:
            assert y_prev is not None, "position restored from an empty cache"
            out[i] = y_prev[i]
    for qi, lst in need.items():
        X = xf[np.asarray(seqs[qi], dtype=np.int64)]
        rows = [j for _, j in lst]
        Y = O.attention_rows(X, W64["wq"], W64["wk"], W64["wv"], W64["wo"], osh.heads, osh.head_dim, rows)
        for (i, _), yrow in zip(lst, Y):
            out[i] = yrow
    return out


def check_layer_step_sampled(x64, W64, osh, ocf, valid, y, tr, positions, y_prev, dtype):
    """Checks one finished call of a layer too large for the full oracle:
    decisions and maps in full, outputs at the sampled positions.  Returns
    the oracle values there and statistics."""
    x64 = np.asarray(x64, dtype=np.float64).reshape(osh.F, osh.N, osh.C)
    dec, _, st = decision_parity(x64, osh, ocf, tr, valid)
    seqs = O.build_sequences(osh, ocf, dec)
    kept_idx, cached_idx, rmap = O.kept_and_map(osh, ocf, dec, seqs, valid)
    check_maps(tr, kept_idx, cached_idx, rmap)
    ref = sampled_outputs(x64, W64, osh, seqs, kept_idx, rmap, positions, y_prev)
    got = to_f64(y).reshape(-1, osh.C)[positions]
    err, raw = rel_err(got, ref, dtype), rel_err(got, ref)
    check_output_bars(err, raw, dtype, "sampled layer output")
    st.update(err=err, err_raw=raw, n_kept=len(kept_idx), n_seq=len(seqs))
    return ref, st


def layer_step_sampled_parity(wl, x_np, sh, cf, osh, ocf, cache, ws, valid, W, W64, positions, y_prev):
    """One oc_layer_cached step of a layer too large for the full oracle."""
    x = dev_tensor(wl, x_np)
    y, _, tr = oc.layer_cached(x, W, cache, sh, cf, ws=ws, trace=True)
    torch.cuda.synchronize()
    return check_layer_step_sampled(wl.f64(x_np), W64, osh, ocf, valid, y, tr, positions, y_prev, wl.dtype)
