"""OmniCache oracle: a plain, slow, single-threaded fp64 reference of one cached
attention layer (Token Cache, Frame Cache, Block Cache; OmniCache §3.2 and
§3.3).

TEST INFRASTRUCTURE ONLY: used by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.  It shares no code
with the HIP library.

Inputs are the exact values of the stored tensors (bf16 or fp32), upcast to
fp64; nothing is rounded afterwards.  Every step follows the paper's order:
descriptors -> cosine similarity -> best match per candidate -> the r most
redundant candidates are cached -> attention over the retained tokens ->
restoration of cached positions -> layer cache update.

Where the paper leaves a choice open, this module takes the following
readings (the same list, with reasons, is kept with the design notes):

  R1  Representative of a 2x2 window: its top-left token (even y, even x).
  R2  Each candidate is compared with every representative of its group.
  R3  A ratio is a fraction of all items of a group, floored (with a 1e-9
      guard) and clamped to the number of candidates.
  R4  Frame Cache: odd frames are candidates, even frames representatives.
  R6  The descriptor of an item is the layer input itself.
  R7  A zero-norm descriptor has similarity 0 with everything.
  R8  Ties: argmax -> smallest representative id; selection -> smallest
      candidate id.
  R9  With no valid cache (first step), a cached position takes the fresh
      output of its matched representative ("matched" cold policy), or the
      step runs with nothing cached ("full" cold policy).
  R10 The cache holds the attention sublayer output (after the output
      projection) at every position and is refreshed every step.
  R11 Cached tokens are neither queries nor keys/values.
  R12 A frame pair caches n_f + floor(r n_f) of its 2 n_f tokens (n_f tokens
      of one frame-patch), clamped to its candidates.
  R13 A 2x2x2 cube of a pair has one representative: the top-left token in
      the pair's representative frame.
  R14 Selected frames are paired greedily, one to one, in selection order.
  R15 The retained tokens of a pair form one attention sequence.
  R16 Text-context tokens are appended to the (single) image sequence and
      never cached.
  R17 Frame Cache with k x k patches (§3.3: the frames are cut into k x k
      patches and the frame set of every patch is matched on its own, the
      batch becoming B*k*k): each patch is a group whose items are the
      frames' tiles of that patch (a tile's descriptor is its tokens'
      features in row-major order, its id the global id of its top-left
      token); odd frames' tiles are candidates, even frames' tiles
      representatives, and each patch caches R = min(floor(r_f F), F/2)
      tiles.  The tokens of a cached tile skip the spatial layer; each
      frame's retained tokens form its attention sequence, whose length
      varies from frame to frame (it may be empty).  k = 1 is the whole-frame
      Frame Cache.
  R20 In a spatial + temporal block the temporal layer's input is the
      residual x + y_spatial; each layer has its own weights and its own
      layer cache (Frame / Token Cache on the spatial layer, Block Cache on
      the temporal one, §3.2).
  R21 The feed-forward sublayer (cached under the same selection as the
      attention of its block, as the SD3 experiments do, §4.2 "Design
      choices") is two linear maps with a tanh-approximated GELU between
      them and no bias: y = GELU(x W1^T) W2^T, W1 [hidden, C], W2 [C,
      hidden].  Retained positions are computed; cached positions keep the
      previous step's FFN output at the same position, or, on a step with
      no valid cache under the "matched" policy, the fresh output of the
      position their best match occupies (the attention call's restore map).
  R23 The hierarchy of §3.3 as a second level for Token and Block Cache:
      coarse_k (dividing patch_k, smaller) and its own ratio r_coarse; its
      groups are the coarse_k x coarse_k patches, their candidates the
      candidates the first level left, their representatives the same
      top-left items; each caches min(floor(r_coarse items), remaining) by
      the usual rule, and a token cached at either level is restored from
      its match at that level.
  (R22, the Layered Cache proposal of Alg. 1, lives in oracle/layered.py.)

Parity unpinned: the frame-pair budget (R12) and the greedy pairing (R14)
have no example in the paper; they are checked by invariants and by an
independent restatement of the greedy (oracle/brute.py) only.

Group order (used to lay out per-candidate results):
  token        : frame-major, then k x k patches row-major
  block        : patches row-major
  frame        : a single group
  frame_token  : attention units (pairs and unmatched frames) ordered by
                 their smallest frame, then patches row-major
Candidates inside a group are listed in ascending id.

Sequences (rows of the reduced attention batch) are ordered by the smallest
item id they cover; inside a sequence, tokens are in ascending global id,
except block sequences, which list frames in ascending order.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

TOKEN, FRAME, BLOCK, FRAME_TOKEN = "token", "frame", "block", "frame_token"
COLD_MATCHED, COLD_FULL = "matched", "full"
FLOOR_GUARD = 1e-9

__all__ = [
    "TOKEN", "FRAME", "BLOCK", "FRAME_TOKEN", "COLD_MATCHED", "COLD_FULL",
    "LayerShape", "CacheCfg", "Group", "Decisions", "StepResult",
    "cosine", "cosine_matrix", "best_match", "skip_count", "pair_skip_count",
    "select_cached", "pair_frames", "token_groups", "block_groups",
    "frame_group", "pair_token_groups", "decide", "build_sequences",
    "kept_and_map", "multi_head_attention", "attn_reduced", "restore",
    "layer_step", "full_attention", "descriptors", "flatten_match",
    "gelu_tanh", "feed_forward", "ffn_step", "block_step", "frame_patch_groups", "tile_tokens",
    "tile_descriptors", "attn_reduced_varlen",
]


# ----------------------------------------------------------------------------
# problem statement
# ----------------------------------------------------------------------------

@dataclass(frozen=True)
class LayerShape:
    """Token tensor [F, N=H*W, C] of one attention layer (OmniCache §3.2.1 and
    §3.2.2 state the (B, T, H, W, C) feature map; B=1 here) plus the layer's
    heads, head dimension and appended uncached context tokens."""
    F: int
    H: int
    W: int
    C: int
    heads: int
    head_dim: int
    n_ctx: int = 0

    @property
    def N(self) -> int:
        return self.H * self.W


@dataclass(frozen=True)
class CacheCfg:
    gran: str                 # token | frame | block | frame_token
    r: float = 0.0            # token (r_t) or block (r_b) ratio
    r_frame: float = 0.0      # frame ratio r_f
    patch_k: int = 1          # k x k patch-local matching (§3.3)
    cold: str = COLD_MATCHED  # reading R9
    coarse_k: int = 0         # second, coarser level of the hierarchy (R23): 0 none
    r_coarse: float = 0.0     # its ratio


@dataclass
class Group:
    """One matching group: representatives (dst) are always retained,
    candidates (src) may be cached.  Ids are token ids (token / pair
    groups), spatial positions (block groups) or frame indices (frame
    group)."""
    items: List[int]
    dst: List[int]
    src: List[int]
    R: int
    kind: str  # "token", "block", "frame"


@dataclass
class Decisions:
    groups: List[Group]
    node_max: List[np.ndarray]      # per group, per candidate
    node_idx: List[np.ndarray]      # per group, per candidate (global rep id)
    cached: List[List[int]]         # per group, cached candidate ids (ascending)
    # frame stage of frame_token (and the frame group of gran=frame)
    frame_group: Optional[Group] = None
    frame_max: Optional[np.ndarray] = None
    frame_idx: Optional[np.ndarray] = None
    frame_cached_order: Optional[List[int]] = None   # selection order
    pairs: Optional[List[Tuple[int, int]]] = None    # (candidate s, rep d)
    frame_sim: Optional[np.ndarray] = None           # [n_src, n_dst] frames


@dataclass
class StepResult:
    y: np.ndarray                 # [F, N, C] layer output after restoration
    y_ctx: Optional[np.ndarray]   # [n_ctx, C]
    y_kept: np.ndarray            # [n_rows, C]
    kept_idx: np.ndarray          # [n_rows] global token ids in row order
    cached_idx: np.ndarray        # ascending cached token ids
    restore_map: np.ndarray       # [F*N]
    sequences: List[List[int]]
    decisions: Decisions


# ----------------------------------------------------------------------------
# similarity and matching (§3.2.1-§3.2.3: cosine-similarity matching)
# ----------------------------------------------------------------------------

def cosine(u: np.ndarray, v: np.ndarray) -> float:
    """Cosine similarity <u,v>/(|u||v|); 0 when either norm is 0 (R7)."""
    nu = math.sqrt(float(np.dot(u, u)))
    nv = math.sqrt(float(np.dot(v, v)))
    if nu == 0.0 or nv == 0.0:
        return 0.0
    return float(np.dot(u, v)) / (nu * nv)


def cosine_matrix(U: np.ndarray, V: np.ndarray) -> np.ndarray:
    """All cosine similarities between rows of U and rows of V (fp64), the
    same definition as ``cosine`` with a library matrix product."""
    U = np.asarray(U, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    nu = np.sqrt(np.einsum("ij,ij->i", U, U))
    nv = np.sqrt(np.einsum("ij,ij->i", V, V))
    dots = U @ V.T
    denom = np.outer(nu, nv)
    out = np.zeros_like(dots)
    ok = denom > 0.0
    out[ok] = dots[ok] / denom[ok]
    return out


def best_match(S: np.ndarray, dst_ids: Sequence[int]) -> Tuple[np.ndarray, np.ndarray]:
    """Per candidate row of S: the largest similarity to any representative
    and the smallest representative id attaining it (R8)."""
    dst_ids = np.asarray(dst_ids, dtype=np.int64)
    assert np.all(np.diff(dst_ids) > 0), "representatives must be listed in ascending id"
    if S.shape[1] == 0:
        return (np.full(S.shape[0], -np.inf), np.full(S.shape[0], -1, dtype=np.int64))
    col = np.argmax(S, axis=1)                 # first (smallest id) maximum
    nmax = S[np.arange(S.shape[0]), col]
    return nmax, dst_ids[col]


# ----------------------------------------------------------------------------
# skip counts and selection
# ----------------------------------------------------------------------------

def skip_count(ratio: float, n_items: int, n_src: int) -> int:
    """Number of candidates to cache in a group: floor(ratio * n_items),
    clamped to the candidate count (R3)."""
    return min(int(math.floor(ratio * n_items + FLOOR_GUARD)), n_src)


def pair_skip_count(ratio: float, n_f: int, n_src: int) -> int:
    """Frame-pair budget (R12): n_f + floor(ratio * n_f), clamped."""
    return min(n_f + int(math.floor(ratio * n_f + FLOOR_GUARD)), n_src)


def selection_order(node_max: Sequence[float], src_ids: Sequence[int]) -> List[int]:
    """Candidate ids sorted from most to least redundant: by decreasing
    best-match similarity, ties by increasing id (R8)."""
    keyed = sorted(zip((-float(v) for v in node_max), (int(i) for i in src_ids)))
    return [i for _, i in keyed]


def select_cached(node_max: Sequence[float], src_ids: Sequence[int], R: int) -> List[int]:
    """The R most redundant candidates (§3.2.1 "the r_b most redundant
    blocks", §3.2.2 "the r_f most redundant frames", §3.2.3 "the r_t most
    redundant positions"), returned in ascending id."""
    return sorted(selection_order(node_max, src_ids)[:R])


# ----------------------------------------------------------------------------
# groups
# ----------------------------------------------------------------------------

def _patches(H: int, W: int, k: int):
    """k x k patch-local scopes (§3.3): lists of (y, x) per patch, row-major."""
    h, w = H // k, W // k
    for py in range(k):
        for px in range(k):
            yield [(y, x) for y in range(py * h, (py + 1) * h)
                   for x in range(px * w, (px + 1) * w)]


def _is_rep(y: int, x: int) -> bool:
    return y % 2 == 0 and x % 2 == 0     # R1


def token_groups(shape: LayerShape, k: int, frames: Sequence[int], ratio: float) -> List[Group]:
    """Token Cache groups of unmatched frames (§3.2.3): per frame and patch,
    2x2 neighbourhoods with the top-left token retained."""
    N, W = shape.N, shape.W
    out = []
    for f in frames:
        for pos in _patches(shape.H, shape.W, k):
            items = sorted(f * N + y * W + x for (y, x) in pos)
            dst = sorted(f * N + y * W + x for (y, x) in pos if _is_rep(y, x))
            src = sorted(f * N + y * W + x for (y, x) in pos if not _is_rep(y, x))
            out.append(Group(items, dst, src, skip_count(ratio, len(items), len(src)), "token"))
    return out


def block_groups(shape: LayerShape, k: int, ratio: float) -> List[Group]:
    """Block Cache groups (§3.2.1): blocks are the per-position temporal
    sequences; 2x2 groups of blocks keep their top-left block."""
    W = shape.W
    out = []
    for pos in _patches(shape.H, shape.W, k):
        items = sorted(y * W + x for (y, x) in pos)
        dst = sorted(y * W + x for (y, x) in pos if _is_rep(y, x))
        src = sorted(y * W + x for (y, x) in pos if not _is_rep(y, x))
        out.append(Group(items, dst, src, skip_count(ratio, len(items), len(src)), "block"))
    return out


def frame_group(shape: LayerShape, ratio: float) -> Group:
    """Frame Cache (§3.2.2): alternating candidate sets, odd frames are
    candidates and even frames representatives (R4)."""
    items = list(range(shape.F))
    dst = [f for f in items if f % 2 == 0]
    src = [f for f in items if f % 2 == 1]
    return Group(items, dst, src, skip_count(ratio, len(items), len(src)), "frame")


def frame_patch_groups(shape: LayerShape, k: int, ratio: float) -> List[Group]:
    """Frame Cache on k x k patches (R17): one group per patch, items are the
    frames' tiles of the patch identified by their top-left token."""
    N, W = shape.N, shape.W
    h, w = shape.H // k, shape.W // k
    out = []
    for py in range(k):
        for px in range(k):
            tl = py * h * W + px * w
            items = [f * N + tl for f in range(shape.F)]
            dst = [f * N + tl for f in range(shape.F) if f % 2 == 0]
            src = [f * N + tl for f in range(shape.F) if f % 2 == 1]
            out.append(Group(items, dst, src, skip_count(ratio, shape.F, len(src)), "frame_patch"))
    return out


def tile_tokens(shape: LayerShape, k: int, tl: int) -> List[int]:
    """Global ids of the tokens of the k x k patch tile whose top-left token
    is tl, in row-major order."""
    N, W = shape.N, shape.W
    h, w = shape.H // k, shape.W // k
    f, n = divmod(tl, N)
    y0, x0 = divmod(n, W)
    return [f * N + (y0 + y) * W + (x0 + x) for y in range(h) for x in range(w)]


def pair_token_groups(shape: LayerShape, k: int, s: int, d: int, ratio: float) -> List[Group]:
    """Token Cache inside a matched frame pair (§3.2.3): the two frames' tokens
    of a patch form one group; each 2x2x2 cube keeps the top-left token of
    the representative frame d (R13); budget per R12."""
    N, W = shape.N, shape.W
    out = []
    for pos in _patches(shape.H, shape.W, k):
        n_f = len(pos)
        items = sorted([s * N + y * W + x for (y, x) in pos] + [d * N + y * W + x for (y, x) in pos])
        dst = sorted(d * N + y * W + x for (y, x) in pos if _is_rep(y, x))
        dset = set(dst)
        src = [i for i in items if i not in dset]
        out.append(Group(items, dst, src, pair_skip_count(ratio, n_f, len(src)), "token"))
    return out


# ----------------------------------------------------------------------------
# descriptors (R6: the layer input itself)
# ----------------------------------------------------------------------------

def descriptors(x: np.ndarray, kind: str, ids: Sequence[int]) -> np.ndarray:
    """x is [F, N, C] fp64.  token: the C-vector of a token; block: the F*C
    concatenation of a position over frames (§3.2.1 reshape to
    (B, H*W, T*C)); frame: the N*C flattening of a frame (§3.2.2 reshape to
    (B, T, H*W*C))."""
    F, N, C = x.shape
    ids = list(ids)
    if kind == "token":
        return x.reshape(F * N, C)[ids]
    if kind == "block":
        return np.stack([x[:, n, :].reshape(F * C) for n in ids]) if ids else np.zeros((0, F * C))
    if kind == "frame":
        return np.stack([x[f].reshape(N * C) for f in ids]) if ids else np.zeros((0, N * C))
    raise ValueError(kind)


def tile_descriptors(x: np.ndarray, shape: LayerShape, k: int, ids: Sequence[int]) -> np.ndarray:
    """Frame-patch tiles (R17): the tile's tokens' features concatenated in
    row-major order."""
    xf = x.reshape(-1, x.shape[-1])
    return np.stack([xf[tile_tokens(shape, k, t)].reshape(-1) for t in ids]) if len(ids) else \
        np.zeros((0, x.shape[-1]))


def _match_group(x: np.ndarray, g: Group, shape: Optional[LayerShape] = None, k: int = 1):
    if g.kind == "frame_patch":
        S = cosine_matrix(tile_descriptors(x, shape, k, g.src), tile_descriptors(x, shape, k, g.dst))
    else:
        S = cosine_matrix(descriptors(x, g.kind, g.src), descriptors(x, g.kind, g.dst))
    return S, best_match(S, g.dst)


# ----------------------------------------------------------------------------
# frame pairing (R14)
# ----------------------------------------------------------------------------

def pair_frames(selected_in_order: Sequence[int], sim: np.ndarray,
                src: Sequence[int], dst: Sequence[int]) -> List[Tuple[int, int]]:
    """Each selected candidate frame, in selection order, takes the free
    representative frame it is most similar to (ties: smallest frame)."""
    src_pos = {f: i for i, f in enumerate(src)}
    taken = set()
    pairs = []
    for s in selected_in_order:
        best = None
        for j, d in enumerate(dst):
            if d in taken:
                continue
            if best is None or sim[src_pos[s], j] > sim[src_pos[s], best]:
                best = j
        taken.add(dst[best])
        pairs.append((s, dst[best]))
    return pairs


# ----------------------------------------------------------------------------
# decisions: match + select (+ pairing)
# ----------------------------------------------------------------------------

def _units(shape: LayerShape, pairs: Sequence[Tuple[int, int]]) -> List[Tuple[int, ...]]:
    """Attention units of frame_token mode: each pair (s, d) and each frame in
    no pair, ordered by their smallest frame."""
    in_pair = set()
    for s, d in pairs:
        in_pair.update((s, d))
    units = [tuple(p) for p in pairs] + [(f,) for f in range(shape.F) if f not in in_pair]
    return sorted(units, key=lambda u: min(u))


def decide(x: np.ndarray, shape: LayerShape, cfg: CacheCfg, no_skip: bool = False,
           forced: Optional[dict] = None) -> Decisions:
    """Matching and selection for one layer call.  ``no_skip`` sets every
    budget to 0 (the "full" cold policy).  ``forced`` may override, for
    parity tests only, decisions that the oracle itself places inside its
    ambiguity band: keys "frame_order" (selected frames in selection order),
    "pairs", "cached" (set of cached item ids), "match" (item -> rep id),
    and with a second level "cached_first" (the first level's cached set
    only, the second level then decided from what it left)."""
    forced = forced or {}
    ratio = 0.0 if no_skip else cfg.r
    fratio = 0.0 if no_skip else cfg.r_frame
    k = cfg.patch_k
    dec_frame = dict()

    if cfg.gran == TOKEN:
        groups = token_groups(shape, k, range(shape.F), ratio)
    elif cfg.gran == BLOCK:
        groups = block_groups(shape, k, ratio)
    elif cfg.gran == FRAME and k > 1:
        groups = frame_patch_groups(shape, k, fratio)
    elif cfg.gran == FRAME:
        groups = [frame_group(shape, fratio)]
    elif cfg.gran == FRAME_TOKEN:
        fg = frame_group(shape, fratio)
        S, (fmax, fidx) = _match_group(x, fg)
        order = selection_order(fmax, fg.src)[:fg.R]
        if "frame_order" in forced:
            order = list(forced["frame_order"])
            assert len(order) == fg.R
        pairs = pair_frames(order, S, fg.src, fg.dst)
        if "pairs" in forced:
            pairs = [tuple(p) for p in forced["pairs"]]
        groups = []
        for u in _units(shape, pairs):
            if len(u) == 2:
                groups += pair_token_groups(shape, k, u[0], u[1], ratio)
            else:
                groups += token_groups(shape, k, [u[0]], ratio)
        dec_frame = dict(frame_group=fg, frame_max=fmax, frame_idx=fidx,
                         frame_cached_order=order, pairs=pairs, frame_sim=S)
    else:
        raise ValueError(cfg.gran)

    node_max, node_idx, cached = [], [], []

    def match_and_select(level_groups, kk):
        for g in level_groups:
            if len(g.src) == 0:
                nm, ni = np.zeros(0), np.zeros(0, dtype=np.int64)
            else:
                _, (nm, ni) = _match_group(x, g, shape, kk)
            node_max.append(nm)
            node_idx.append(np.asarray(ni, dtype=np.int64))
            cached.append(select_cached(nm, g.src, g.R))

    match_and_select(groups, k)
    if cfg.coarse_k:
        force = forced.get("cached")
        first = forced.get("cached_first", force)
        if first is not None:
            # a forced selection fixes the first level before the second is
            # formed from what it left ("cached_first": the first level only)
            cached = [_forced_in(g, first) for g in groups]
        n1 = len(groups)
        groups = groups + coarse_groups(shape, cfg, set(i for c in cached for i in c),
                                        0.0 if no_skip else cfg.r_coarse)
        match_and_select(groups[n1:], cfg.coarse_k)
        if force is not None:
            cached = cached[:n1] + [_forced_in(g, force) for g in groups[n1:]]
        dec = Decisions(groups, node_max, node_idx, cached, **dec_frame)
        return force_decisions(dec, None, forced.get("match"))
    dec = Decisions(groups, node_max, node_idx, cached, **dec_frame)
    return force_decisions(dec, forced.get("cached"), forced.get("match"))


def _forced_in(g: Group, cached: set) -> List[int]:
    c = sorted(i for i in g.src if i in cached)
    assert len(c) == g.R, "forced selection must keep the group's budget"
    return c


def coarse_groups(shape: LayerShape, cfg: CacheCfg, cached_first: set, ratio: float) -> List[Group]:
    """The second, coarser level of the hierarchy (§3.3, reading R23): the
    groups of coarse_k x coarse_k patches, each a union of first-level
    patches; their candidates are those the first level did not cache,
    their representatives the same top-left items, and each caches
    min(floor(r_coarse * items), remaining candidates)."""
    if cfg.gran not in (TOKEN, BLOCK):
        raise ValueError("a coarser level is defined for Token and Block Cache")
    if not (1 <= cfg.coarse_k < cfg.patch_k and cfg.patch_k % cfg.coarse_k == 0):
        raise ValueError("coarse_k must divide patch_k and be smaller")
    base = token_groups(shape, cfg.coarse_k, range(shape.F), ratio) if cfg.gran == TOKEN else \
        block_groups(shape, cfg.coarse_k, ratio)
    out = []
    for g in base:
        rest = [i for i in g.src if i not in cached_first]
        out.append(Group(g.items, g.dst, rest, skip_count(ratio, len(g.items), len(rest)), g.kind))
    return out


def force_decisions(dec: Decisions, cached: Optional[set] = None, match: Optional[dict] = None) -> Decisions:
    """The decisions with, for parity tests only, some candidates' matched
    representative (``match``: item -> rep id) and the cached set of every
    group (``cached``: item ids, the group's budget kept) replaced."""
    if cached is None and not match:
        return dec
    match = match or {}
    node_idx = [np.array([match.get(int(s), int(v)) for s, v in zip(g.src, ni)], dtype=np.int64)
                for g, ni in zip(dec.groups, dec.node_idx)]
    sel = dec.cached
    if cached is not None:
        sel = []
        for g in dec.groups:
            c = sorted(i for i in g.src if i in cached)
            assert len(c) == g.R, "forced selection must keep the group's budget"
            sel.append(c)
    return Decisions(dec.groups, dec.node_max, node_idx, sel, dec.frame_group, dec.frame_max, dec.frame_idx,
                     dec.frame_cached_order, dec.pairs, dec.frame_sim)


# ----------------------------------------------------------------------------
# sequences, kept rows and the restore map
# ----------------------------------------------------------------------------

def build_sequences(shape: LayerShape, cfg: CacheCfg, dec: Decisions) -> List[List[int]]:
    """Retained tokens grouped into attention sequences (§3.2.1: blocks are
    per-position temporal sequences; §3.2.2/§3.2.3: spatial sequences per
    frame or per matched pair, R15)."""
    F, N = shape.F, shape.N
    cached_items = set(i for c in dec.cached for i in c)
    if cfg.gran == TOKEN:
        return [[f * N + n for n in range(N) if f * N + n not in cached_items] for f in range(F)]
    if cfg.gran == FRAME and cfg.patch_k > 1:
        dropped = set(p for t in cached_items for p in tile_tokens(shape, cfg.patch_k, t))
        return [[f * N + n for n in range(N) if f * N + n not in dropped] for f in range(F)]
    if cfg.gran == FRAME:
        return [[f * N + n for n in range(N)] for f in range(F) if f not in cached_items]
    if cfg.gran == BLOCK:
        return [[f * N + n for f in range(F)] for n in range(N) if n not in cached_items]
    if cfg.gran == FRAME_TOKEN:
        seqs = []
        for u in _units(shape, dec.pairs):
            toks = sorted(f * N + n for f in u for n in range(N))
            seqs.append([p for p in toks if p not in cached_items])
        return seqs
    raise ValueError(cfg.gran)


def matched_token(shape: LayerShape, cfg: CacheCfg, dec: Decisions) -> Dict[int, int]:
    """For every cached token position, the token whose fresh output replaces
    it under the "matched" cold policy (R9): the matched representative
    token; for a cached frame f matched to frame d, token (d, n); for a
    cached block n matched to block m, token (f, m)."""
    F, N = shape.F, shape.N
    out = {}
    for g, ni, c in zip(dec.groups, dec.node_idx, dec.cached):
        rep_of = {int(s): int(d) for s, d in zip(g.src, ni)}
        for item in c:
            rep = rep_of[item]
            if g.kind == "token":
                out[item] = rep
            elif g.kind == "frame":
                for n in range(N):
                    out[item * N + n] = rep * N + n
            elif g.kind == "block":
                for f in range(F):
                    out[f * N + item] = f * N + rep
            elif g.kind == "frame_patch":
                d = rep // N                       # token n of the tile takes token n of frame d
                for p in tile_tokens(shape, cfg.patch_k, item):
                    out[p] = d * N + p % N
    return out


def kept_and_map(shape: LayerShape, cfg: CacheCfg, dec: Decisions, seqs: List[List[int]],
                 cache_valid: bool) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """kept_idx (row -> token), cached_idx (ascending) and the restore map:
    map[p] = row of p if p is retained; -1 if p is restored from the cache
    (valid cache); else the row of p's matched representative (R9)."""
    kept = [p for s in seqs for p in s]
    row_of = {p: i for i, p in enumerate(kept)}
    FN = shape.F * shape.N
    cached_tokens = sorted(p for p in range(FN) if p not in row_of)
    rmap = np.full(FN, -1, dtype=np.int64)
    for p, i in row_of.items():
        rmap[p] = i
    if not cache_valid and cached_tokens:
        mt = matched_token(shape, cfg, dec)
        for p in cached_tokens:
            rmap[p] = row_of[mt[p]]
    return np.array(kept, dtype=np.int64), np.array(cached_tokens, dtype=np.int64), rmap


# ----------------------------------------------------------------------------
# attention over the retained tokens (R11)
# ----------------------------------------------------------------------------

def multi_head_attention(X: np.ndarray, wq: np.ndarray, wk: np.ndarray, wv: np.ndarray,
                         wo: np.ndarray, heads: int, head_dim: int) -> np.ndarray:
    """Plain multi-head self-attention of one sequence X [L, C]:
    Q = X Wq^T, K = X Wk^T, V = X Wv^T (weights in out x in layout), per head
    softmax(Q_h K_h^T / sqrt(head_dim)) V_h with the row maximum subtracted,
    heads concatenated, then the output projection Wo^T.  No bias,
    normalisation or positional term."""
    Q = X @ wq.T
    K = X @ wk.T
    V = X @ wv.T
    O = np.empty_like(Q)
    scale = 1.0 / math.sqrt(head_dim)
    for h in range(heads):
        sl = slice(h * head_dim, (h + 1) * head_dim)
        s = (Q[:, sl] @ K[:, sl].T) * scale
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=1, keepdims=True)
        O[:, sl] = p @ V[:, sl]
    return O @ wo.T


def attention_rows(X: np.ndarray, wq: np.ndarray, wk: np.ndarray, wv: np.ndarray, wo: np.ndarray,
                   heads: int, head_dim: int, rows: Sequence[int]) -> np.ndarray:
    """The rows ``rows`` of multi_head_attention(X, ...): the same definition
    with the queries restricted to those tokens, keys and values over all of
    X.  Lets a check of a very long sequence compute a sample of outputs."""
    rows = np.asarray(rows, dtype=np.int64)
    Q = X[rows] @ wq.T
    K = X @ wk.T
    V = X @ wv.T
    O = np.empty_like(Q)
    scale = 1.0 / math.sqrt(head_dim)
    for h in range(heads):
        sl = slice(h * head_dim, (h + 1) * head_dim)
        s = (Q[:, sl] @ K[:, sl].T) * scale
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=1, keepdims=True)
        O[:, sl] = p @ V[:, sl]
    return O @ wo.T


def attn_reduced(x_kept: np.ndarray, ctx: Optional[np.ndarray], w: Dict[str, np.ndarray],
                 heads: int, head_dim: int) -> Tuple[np.ndarray, Optional[np.ndarray]]:
    """x_kept is [n_seq, L, C]; each sequence attends within itself, with the
    context tokens appended when given (only for a single sequence, R16).
    Returns y_kept [n_seq*L, C] and y_ctx [n_ctx, C] (or None)."""
    n_seq, L, C = x_kept.shape
    ys = []
    y_ctx = None
    for q in range(n_seq):
        X = x_kept[q]
        if ctx is not None and len(ctx):
            assert n_seq == 1
            X = np.concatenate([X, ctx], axis=0)
        Y = multi_head_attention(X, w["wq"], w["wk"], w["wv"], w["wo"], heads, head_dim)
        ys.append(Y[:L])
        if ctx is not None and len(ctx):
            y_ctx = Y[L:]
    y_kept = np.concatenate(ys, axis=0) if ys else np.zeros((0, C))
    return y_kept, y_ctx


def attn_reduced_varlen(xs: Sequence[np.ndarray], w: Dict[str, np.ndarray], heads: int,
                        head_dim: int) -> np.ndarray:
    """Sequences of different lengths (R17), each attending within itself;
    rows of all sequences concatenated in sequence order.  An empty
    sequence contributes no rows."""
    C = w["wo"].shape[0]
    ys = [multi_head_attention(X, w["wq"], w["wk"], w["wv"], w["wo"], heads, head_dim) for X in xs if len(X)]
    return np.concatenate(ys, axis=0) if ys else np.zeros((0, C))


# ----------------------------------------------------------------------------
# restoration and the layer step
# ----------------------------------------------------------------------------

def restore(y_kept: np.ndarray, restore_map: np.ndarray, cache_y: Optional[np.ndarray]) -> np.ndarray:
    """Cached positions are restored at their original location (§3.2.1
    "restores cached blocks to their original spatial positions", §3.2.3
    "scattered back to the original frame layout"): y[p] = y_kept[map[p]]
    when map[p] >= 0, else the cached activation at the same position."""
    FN = restore_map.shape[0]
    C = y_kept.shape[1]
    y = np.empty((FN, C), dtype=np.float64)
    for p in range(FN):
        m = int(restore_map[p])
        y[p] = y_kept[m] if m >= 0 else cache_y[p]
    return y


def layer_step(x: np.ndarray, ctx: Optional[np.ndarray], w: Dict[str, np.ndarray],
               shape: LayerShape, cfg: CacheCfg, cache_y: Optional[np.ndarray],
               cache_valid: bool, forced: Optional[dict] = None) -> StepResult:
    """One cached layer call: decisions, reduced attention, restoration.  The
    caller keeps ``y`` as the next step's cache (R10)."""
    x = np.asarray(x, dtype=np.float64).reshape(shape.F, shape.N, shape.C)
    no_skip = (not cache_valid) and cfg.cold == COLD_FULL
    dec = decide(x, shape, cfg, no_skip=no_skip, forced=forced)
    seqs = build_sequences(shape, cfg, dec)
    kept_idx, cached_idx, rmap = kept_and_map(shape, cfg, dec, seqs, cache_valid)
    xf = x.reshape(shape.F * shape.N, shape.C)
    lens = {len(s) for s in seqs}
    c64 = None if ctx is None else np.asarray(ctx, dtype=np.float64)
    if len(lens) <= 1:
        L = lens.pop() if lens else 0
        x_kept = xf[kept_idx].reshape(len(seqs), L, shape.C)
        y_kept, y_ctx = attn_reduced(x_kept, c64, w, shape.heads, shape.head_dim)
    else:
        # Frame Cache on patches (R17): sequences of different lengths
        assert cfg.gran == FRAME and cfg.patch_k > 1 and c64 is None
        y_kept = attn_reduced_varlen([xf[np.asarray(sq, dtype=np.int64)] for sq in seqs], w, shape.heads,
                                     shape.head_dim)
        y_ctx = None
    cy = None if cache_y is None else np.asarray(cache_y, dtype=np.float64).reshape(-1, shape.C)
    y = restore(y_kept, rmap, cy)
    return StepResult(y.reshape(shape.F, shape.N, shape.C), y_ctx, y_kept, kept_idx,
                      cached_idx, rmap, seqs, dec)


def full_attention(x: np.ndarray, ctx: Optional[np.ndarray], w: Dict[str, np.ndarray],
                   shape: LayerShape, temporal: bool = False) -> Tuple[np.ndarray, Optional[np.ndarray]]:
    """The uncached layer: spatial attention per frame over all its tokens
    (+ context), or temporal attention per position over all frames."""
    x = np.asarray(x, dtype=np.float64).reshape(shape.F, shape.N, shape.C)
    y = np.empty_like(x)
    y_ctx = None
    c64 = None if ctx is None else np.asarray(ctx, dtype=np.float64)
    if temporal:
        for n in range(shape.N):
            y[:, n, :] = multi_head_attention(x[:, n, :], w["wq"], w["wk"], w["wv"], w["wo"],
                                              shape.heads, shape.head_dim)
        return y, None
    for f in range(shape.F):
        X = x[f]
        if c64 is not None and len(c64):
            X = np.concatenate([X, c64], axis=0)
        Y = multi_head_attention(X, w["wq"], w["wk"], w["wv"], w["wo"], shape.heads, shape.head_dim)
        y[f] = Y[:shape.N]
        if c64 is not None and len(c64):
            y_ctx = Y[shape.N:]
    return y, y_ctx


# ----------------------------------------------------------------------------
# helpers for laying results out like the library's per-candidate arrays
# ----------------------------------------------------------------------------

def flatten_match(dec: Decisions) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """[n_groups, n_src_max] arrays of node_max (-inf pad), node_idx (-1 pad)
    and candidate ids (-1 pad), in group order."""
    G = len(dec.groups)
    m = max((len(g.src) for g in dec.groups), default=0)
    nm = np.full((G, m), -np.inf)
    ni = np.full((G, m), -1, dtype=np.int64)
    ids = np.full((G, m), -1, dtype=np.int64)
    for gi, g in enumerate(dec.groups):
        n = len(g.src)
        nm[gi, :n] = dec.node_max[gi]
        ni[gi, :n] = dec.node_idx[gi]
        ids[gi, :n] = g.src
    return nm, ni, ids


# ----------------------------------------------------------------------------
# feed-forward sublayer under the same selection (R21)
# ----------------------------------------------------------------------------

def gelu_tanh(u: np.ndarray) -> np.ndarray:
    """GELU with the tanh approximation:
    0.5 u (1 + tanh(sqrt(2/pi) (u + 0.044715 u^3)))."""
    u = np.asarray(u, dtype=np.float64)
    return 0.5 * u * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (u + 0.044715 * u ** 3)))


def feed_forward(X: np.ndarray, w1: np.ndarray, w2: np.ndarray) -> np.ndarray:
    """The feed-forward map of rows X [n, C]: GELU(X W1^T) W2^T (R21)."""
    return gelu_tanh(X @ w1.T) @ w2.T


def ffn_step(x: np.ndarray, kept_idx: np.ndarray, restore_map: np.ndarray, w1: np.ndarray, w2: np.ndarray,
             cache_y: Optional[np.ndarray]) -> np.ndarray:
    """One cached FFN call under a selection made by the attention sublayer:
    the retained rows x[kept_idx] go through the feed-forward map (row i of
    the reduced batch is token kept_idx[i]) and every position is then
    restored through the same restore map as the attention output (§3.2.3
    restoration at original positions; R9 on a cold step).  x is [F*N, C]."""
    x = np.asarray(x, dtype=np.float64).reshape(-1, w1.shape[1])
    y_kept = feed_forward(x[np.asarray(kept_idx, dtype=np.int64)], w1, w2)
    cy = None if cache_y is None else np.asarray(cache_y, dtype=np.float64).reshape(-1, w1.shape[1])
    return restore(y_kept, np.asarray(restore_map), cy)


# ----------------------------------------------------------------------------
# a spatial + temporal block with all three caches (R20)
# ----------------------------------------------------------------------------

def block_step(x: np.ndarray, w_spatial: Dict[str, np.ndarray], w_temporal: Dict[str, np.ndarray],
               shape: LayerShape, spatial: CacheCfg, temporal: CacheCfg,
               cache_s: Optional[np.ndarray], valid_s: bool, cache_t: Optional[np.ndarray], valid_t: bool,
               forced_s: Optional[dict] = None, forced_t: Optional[dict] = None,
               h: Optional[np.ndarray] = None) -> Tuple[StepResult, np.ndarray, StepResult]:
    """The spatial layer (Frame / Token Cache) on x, the residual
    h = x + y_spatial, then the temporal layer (Block Cache) on h.  ``h``,
    when given, replaces the residual as the temporal layer's input (a
    caller comparing a library that stores h rounded to its tensor type
    passes that stored h, so that each layer is checked on its exact input).
    Returns (spatial result, h, temporal result)."""
    assert temporal.gran == BLOCK and spatial.gran != BLOCK
    rs = layer_step(x, None, w_spatial, shape, spatial, cache_s, valid_s, forced=forced_s)
    hh = np.asarray(x, dtype=np.float64).reshape(rs.y.shape) + rs.y if h is None else \
        np.asarray(h, dtype=np.float64).reshape(rs.y.shape)
    rt = layer_step(hh, None, w_temporal, shape, temporal, cache_t, valid_t, forced=forced_t)
    return rs, hh, rt
