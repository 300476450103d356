"""Seeded synthetic workloads shaped like the attention layers of SD3, Latte
and SVD-XT (OmniCache §4.1 names the models; their weights and datasets are
not used: every tensor here is drawn from a seeded generator).

Recipe (all draws from ``numpy.random.Generator(PCG64(seed))``, fp32):

* A smooth feature field of shape [C, gh, gw] ~ N(0, 1) is upsampled to the
  H x W token grid with bilinear interpolation, half-pixel centres and edge
  clamping.  Tokens are laid out [F, H*W, C], token (f, y, x) at row
  f*H*W + y*W + x.
* Per-workload structure (noise, per-frame cumulative drift, translation) is
  added on top, in the order documented in each builder below.
* Weights are drawn after the activations, in the order q, k, v, o, each
  ~ N(0, 1/C).  They are stored in the out-features x in-features layout of a
  linear layer: wq, wk, wv are [heads*head_dim, C] and wo is [C, heads*head_dim].
* Denoising steps: step s > 0 is step s-1 plus 0.02 * N(0, 1) on the fp32
  master copy (text-context rows, when present, stay fixed).
* bf16 workloads round every tensor once, round-to-nearest-even, from the
  fp32 master.  bf16 tensors are returned as uint16 bit patterns.

Nothing in this module computes any part of the caching method.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np


# ----------------------------------------------------------------------------
# bf16 storage helpers (round-to-nearest-even from fp32)
# ----------------------------------------------------------------------------

def bf16_bits(a: np.ndarray) -> np.ndarray:
    """fp32 array -> uint16 bf16 bit patterns, round to nearest even."""
    b = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    lsb = (b >> np.uint32(16)) & np.uint32(1)
    r = (b + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(u: np.ndarray) -> np.ndarray:
    """uint16 bf16 bit patterns -> exactly equal fp32 values."""
    return (np.ascontiguousarray(u, dtype=np.uint16).astype(np.uint32)
            << np.uint32(16)).view(np.float32)


# ----------------------------------------------------------------------------
# field synthesis
# ----------------------------------------------------------------------------

def _interp_matrix(n_in: int, n_out: int, shift: float = 0.0) -> np.ndarray:
    """Bilinear interpolation weights [n_out, n_in]: half-pixel centres, edge
    clamp.  ``shift`` moves the sampling grid by that many output cells
    (output cell i samples the field at i - shift)."""
    m = np.zeros((n_out, n_in), dtype=np.float64)
    scale = n_in / n_out
    for i in range(n_out):
        src = (i - shift + 0.5) * scale - 0.5
        src = min(max(src, 0.0), n_in - 1.0)
        i0 = int(math.floor(src))
        i1 = min(i0 + 1, n_in - 1)
        w = src - i0
        m[i, i0] += 1.0 - w
        m[i, i1] += w
    return m


def _upsample(field_chw: np.ndarray, H: int, W: int,
              shift_x: float = 0.0) -> np.ndarray:
    """[C, gh, gw] -> [H*W, C] fp32."""
    C, gh, gw = field_chw.shape
    my = _interp_matrix(gh, H)
    mx = _interp_matrix(gw, W, shift_x)
    f64 = field_chw.astype(np.float64)
    t = np.einsum("yi,cij->cyj", my, f64)
    t = np.einsum("xj,cyj->yxc", mx, t)
    return np.ascontiguousarray(t.reshape(H * W, C), dtype=np.float32)


# ----------------------------------------------------------------------------
# workload container
# ----------------------------------------------------------------------------

GRANS = ("token", "frame", "block", "frame_token")


@dataclass
class Workload:
    name: str
    F: int
    H: int
    W: int
    C: int
    heads: int
    head_dim: int
    n_ctx: int
    dtype: str                 # "f32" or "bf16"
    gran: str                  # one of GRANS
    r: float                   # token / block ratio
    r_frame: float             # frame ratio
    patch_k: int
    steps: List[np.ndarray]    # per step [F, H*W, C]: float32, or uint16 bf16 bits
    ctx: Optional[np.ndarray]  # [n_ctx, C] same storage, or None
    wq: np.ndarray             # [heads*head_dim, C]
    wk: np.ndarray
    wv: np.ndarray
    wo: np.ndarray             # [C, heads*head_dim]
    # second (temporal) layer of a spatial+temporal level, when present
    t_weights: Optional[Dict[str, np.ndarray]] = None
    note: str = ""
    extra: Dict[str, object] = field(default_factory=dict)

    @property
    def N(self) -> int:
        return self.H * self.W

    def to_f32(self, a: np.ndarray) -> np.ndarray:
        """Exact fp32 values of a stored tensor."""
        return bf16_bits_to_f32(a) if self.dtype == "bf16" else a

    def f64(self, a: np.ndarray) -> np.ndarray:
        return self.to_f32(a).astype(np.float64)


def _store(a32: np.ndarray, dtype: str) -> np.ndarray:
    return bf16_bits(a32) if dtype == "bf16" else np.ascontiguousarray(a32, np.float32)


def _weights(rng, C, heads, head_dim, dtype):
    hd = heads * head_dim
    s = 1.0 / math.sqrt(C)
    wq = rng.standard_normal((hd, C), dtype=np.float32) * np.float32(s)
    wk = rng.standard_normal((hd, C), dtype=np.float32) * np.float32(s)
    wv = rng.standard_normal((hd, C), dtype=np.float32) * np.float32(s)
    wo = rng.standard_normal((C, hd), dtype=np.float32) * np.float32(s)
    return tuple(_store(w, dtype) for w in (wq, wk, wv, wo))


def _step_chain(rng, x0: np.ndarray, n_steps: int, dtype: str,
                plant=None) -> List[np.ndarray]:
    """Step s = step s-1 + 0.02 N(0,1) on the fp32 master; ``plant`` (if
    given) rewrites the master after each step's drift."""
    out = []
    x = x0
    for s in range(n_steps):
        if s > 0:
            x = x + np.float32(0.02) * rng.standard_normal(x.shape, dtype=np.float32)
        xs = plant(rng, x) if plant is not None else x
        out.append(_store(xs, dtype))
    return out


def _plant_odd_frames(rng, x: np.ndarray) -> np.ndarray:
    """Odd frame 2m+1 := frame 2m + 0.01 (m+1) N(0,1): frame pairs with known,
    well separated similarities."""
    y = x.copy()
    F = x.shape[0]
    for m in range((F) // 2):
        if 2 * m + 1 < F:
            y[2 * m + 1] = x[2 * m] + np.float32(0.01 * (m + 1)) * \
                rng.standard_normal(x.shape[1:], dtype=np.float32)
    return y


# ----------------------------------------------------------------------------
# builders
# ----------------------------------------------------------------------------

def _tok16(n_steps):
    """Token Cache on one 16x16 frame, C=64, one head of 64, fp32, r=0.5:
    upsampled 4x4 field + 0.1 N(0,1)."""
    rng = np.random.Generator(np.random.PCG64(1001))
    F, H, W, C, heads, dh = 1, 16, 16, 64, 1, 64
    fld = rng.standard_normal((C, 4, 4), dtype=np.float32)
    x0 = _upsample(fld, H, W)[None] + np.float32(0.1) * rng.standard_normal((F, H * W, C), dtype=np.float32)
    w = _weights(rng, C, heads, dh, "f32")
    steps = _step_chain(rng, x0, n_steps, "f32")
    return Workload("tok16_f32", F, H, W, C, heads, dh, 0, "f32", "token", 0.5, 0.0, 1,
                    steps, None, *w)


def _sd3(n_steps):
    """SD3-1024-like joint attention layer: 64x64 image tokens + 333 text
    tokens (never cached), C=1536, 24 heads x 64, bf16.  Image tokens =
    upsampled 16x16 field + 0.05 N(0,1); text ~ N(0,1), fixed over steps;
    step drift on image tokens only."""
    rng = np.random.Generator(np.random.PCG64(1002))
    F, H, W, C, heads, dh, nctx = 1, 64, 64, 1536, 24, 64, 333
    fld = rng.standard_normal((C, 16, 16), dtype=np.float32)
    x0 = _upsample(fld, H, W)[None] + np.float32(0.05) * rng.standard_normal((F, H * W, C), dtype=np.float32)
    ctx = rng.standard_normal((nctx, C), dtype=np.float32)
    w = _weights(rng, C, heads, dh, "bf16")
    steps = _step_chain(rng, x0, n_steps, "bf16")
    return Workload("sd3_1024", F, H, W, C, heads, dh, nctx, "bf16", "token", 0.5, 0.0, 1,
                    steps, _store(ctx, "bf16"), *w)


def _latte_frames(rng, F, H, W, C, shift_per_frame=0.0):
    """Shared base (upsampled 8x8 field), optionally translated by
    shift_per_frame tokens per frame along x, + cumulative 0.03 N(0,1) drift
    per frame + 0.02 N(0,1) noise."""
    fld = rng.standard_normal((C, 8, 8), dtype=np.float32)
    x = np.empty((F, H * W, C), dtype=np.float32)
    drift = np.zeros((H * W, C), dtype=np.float32)
    for f in range(F):
        base = _upsample(fld, H, W, shift_x=shift_per_frame * f)
        drift = drift + np.float32(0.03) * rng.standard_normal((H * W, C), dtype=np.float32)
        x[f] = base + drift + np.float32(0.02) * rng.standard_normal((H * W, C), dtype=np.float32)
    return x


def _latte_spatial(n_steps, planted=False):
    """Latte-like spatial layer with Frame Cache: 16 frames of 16x16 tokens,
    C=1152, 16 heads x 72, bf16, frame ratio 0.25."""
    rng = np.random.Generator(np.random.PCG64(1003))
    F, H, W, C, heads, dh = 16, 16, 16, 1152, 16, 72
    x0 = _latte_frames(rng, F, H, W, C)
    w = _weights(rng, C, heads, dh, "bf16")
    steps = _step_chain(rng, x0, n_steps, "bf16", _plant_odd_frames if planted else None)
    name = "latte_spatial_planted" if planted else "latte_spatial"
    return Workload(name, F, H, W, C, heads, dh, 0, "bf16", "frame", 0.0, 0.25, 1,
                    steps, None, *w)


def _latte_temporal(n_steps):
    """Latte-like temporal layer with Block Cache: the spatial generator with a
    smooth translation of 0.5 token per frame; 256 blocks of 16 frames,
    C=1152, 16 heads x 72, bf16, block ratio 0.5."""
    rng = np.random.Generator(np.random.PCG64(1004))
    F, H, W, C, heads, dh = 16, 16, 16, 1152, 16, 72
    x0 = _latte_frames(rng, F, H, W, C, shift_per_frame=0.5)
    w = _weights(rng, C, heads, dh, "bf16")
    steps = _step_chain(rng, x0, n_steps, "bf16")
    return Workload("latte_temporal", F, H, W, C, heads, dh, 0, "bf16", "block", 0.5, 0.0, 1,
                    steps, None, *w)


def _svdxt(n_steps, planted=False, patch_k=1):
    """SVD-XT-like U-Net level: 25 frames of 72x128 tokens, C=320, 5 heads x 64,
    bf16; upsampled 18x32 field + cumulative 0.02 N(0,1) drift per frame +
    0.05 N(0,1) noise.  Spatial layer with Frame+Token Cache (token ratio
    0.5, frame ratio 0.2), followed by an uncached temporal layer with its own
    weights."""
    rng = np.random.Generator(np.random.PCG64(1005))
    F, H, W, C, heads, dh = 25, 72, 128, 320, 5, 64
    fld = rng.standard_normal((C, 18, 32), dtype=np.float32)
    base = _upsample(fld, H, W)
    x0 = np.empty((F, H * W, C), dtype=np.float32)
    drift = np.zeros((H * W, C), dtype=np.float32)
    for f in range(F):
        drift = drift + np.float32(0.02) * rng.standard_normal((H * W, C), dtype=np.float32)
        x0[f] = base + drift + np.float32(0.05) * rng.standard_normal((H * W, C), dtype=np.float32)
    w = _weights(rng, C, heads, dh, "bf16")
    tw = _weights(rng, C, heads, dh, "bf16")
    steps = _step_chain(rng, x0, n_steps, "bf16", _plant_odd_frames if planted else None)
    name = ("svdxt_level_planted" if planted else "svdxt_level") + ("" if patch_k == 1 else f"_k{patch_k}")
    return Workload(name, F, H, W, C, heads, dh, 0, "bf16", "frame_token", 0.5, 0.2, patch_k,
                    steps, None, *w, t_weights=dict(wq=tw[0], wk=tw[1], wv=tw[2], wo=tw[3]))


def _latte_block(n_steps):
    """Latte-like spatial + temporal block with all three caches at the
    paper's Latte ratios (r_f / r_b / r_t = 30 / 40 / 20 %): 16 frames of
    16x16 tokens, C=1152, 16 heads x 72, bf16; the Latte generator with the
    0.5 token-per-frame translation (frame and motion redundancy both
    present); spatial and temporal layers with their own weights."""
    rng = np.random.Generator(np.random.PCG64(1006))
    F, H, W, C, heads, dh = 16, 16, 16, 1152, 16, 72
    x0 = _latte_frames(rng, F, H, W, C, shift_per_frame=0.5)
    w = _weights(rng, C, heads, dh, "bf16")
    tw = _weights(rng, C, heads, dh, "bf16")
    steps = _step_chain(rng, x0, n_steps, "bf16")
    return Workload("latte_block", F, H, W, C, heads, dh, 0, "bf16", "frame_token", 0.2, 0.3, 1,
                    steps, None, *w, t_weights=dict(wq=tw[0], wk=tw[1], wv=tw[2], wo=tw[3]),
                    extra=dict(r_block=0.4, block_patch_k=1))


def _svdxt_block(n_steps):
    """SVD-XT-like spatial + temporal block at the paper's SVD-XT ratios
    (r_f / r_b / r_t = 50 / 40 / 50 %): the SVD-XT-like level's inputs and
    weights, token and block matching patch-local in 4x4 patches (§3.3)."""
    wl = _svdxt(n_steps, patch_k=4)
    wl.name = "svdxt_block"
    wl.r, wl.r_frame = 0.5, 0.5
    wl.extra = dict(r_block=0.4, block_patch_k=4)
    return wl


WORKLOADS = {
    "tok16_f32": _tok16,
    "sd3_1024": _sd3,
    "latte_spatial": _latte_spatial,
    "latte_spatial_planted": lambda n: _latte_spatial(n, planted=True),
    "latte_temporal": _latte_temporal,
    "svdxt_level": _svdxt,
    "svdxt_level_k4": lambda n: _svdxt(n, patch_k=4),
    "svdxt_level_planted": lambda n: _svdxt(n, planted=True),
    "latte_block": _latte_block,
    "svdxt_block": _svdxt_block,
}


def ffn_weights(C: int, hidden: int, dtype: str, seed: int = 2000) -> Dict[str, np.ndarray]:
    """Feed-forward weights of a layer of width C: w1 [hidden, C] ~ N(0, 1/C)
    then w2 [C, hidden] ~ N(0, 1/hidden), drawn from their own seeded
    generator (so adding them leaves every attention workload unchanged)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    w1 = rng.standard_normal((hidden, C), dtype=np.float32) * np.float32(1.0 / math.sqrt(C))
    w2 = rng.standard_normal((C, hidden), dtype=np.float32) * np.float32(1.0 / math.sqrt(hidden))
    return dict(w1=_store(w1, dtype), w2=_store(w2, dtype))


def layered_tables(n_layers: int = 24, n_steps: int = 28, seed: int = 3000):
    """Synthetic per-(layer, timestep) tables for the Layered Cache schedule,
    shaped like SD3-medium (24 transformer blocks, 28 sampling steps; §4.1):
    latency saved by caching a pair ~ 1 ms with 10% spread (blocks of one
    width cost alike), and quality loss log-normal, four times larger in the
    first and last four blocks and larger at early timesteps (§4.2 finds early
    and late layers most sensitive).  Returns (latency, quality), fp64
    [n_layers, n_steps]."""
    rng = np.random.Generator(np.random.PCG64(seed))
    lat = np.clip(1.0 + 0.1 * rng.standard_normal((n_layers, n_steps)), 0.5, None)
    edge = np.array([4.0 if (l < 4 or l >= n_layers - 4) else 1.0 for l in range(n_layers)])
    early = 1.0 + 2.0 * np.exp(-np.arange(n_steps) / 4.0)
    qual = np.exp(0.5 * rng.standard_normal((n_layers, n_steps))) * edge[:, None] * early[None, :]
    return lat, qual


def make_workload(name: str, n_steps: int = 4) -> Workload:
    return WORKLOADS[name](n_steps)


def small_workload(gran: str = "token", F: int = 1, H: int = 8, W: int = 8,
                   C: int = 32, heads: int = 2, head_dim: int = 16,
                   n_ctx: int = 0, dtype: str = "f32", r: float = 0.5,
                   r_frame: float = 0.25, patch_k: int = 1, n_steps: int = 1,
                   seed: int = 7, field_grid: int = 2, noise: float = 0.1,
                   frame_drift: float = 0.03, planted: bool = False) -> Workload:
    """A small workload with the same recipe family: upsampled field + per-frame
    cumulative drift + noise (+ optional planted odd frames)."""
    assert gran in GRANS
    rng = np.random.Generator(np.random.PCG64(seed))
    fld = rng.standard_normal((C, field_grid, field_grid), dtype=np.float32)
    base = _upsample(fld, H, W)
    x0 = np.empty((F, H * W, C), dtype=np.float32)
    drift = np.zeros((H * W, C), dtype=np.float32)
    for f in range(F):
        drift = drift + np.float32(frame_drift) * rng.standard_normal((H * W, C), dtype=np.float32)
        x0[f] = base + drift + np.float32(noise) * rng.standard_normal((H * W, C), dtype=np.float32)
    ctx = rng.standard_normal((n_ctx, C), dtype=np.float32) if n_ctx > 0 else None
    w = _weights(rng, C, heads, head_dim, dtype)
    steps = _step_chain(rng, x0, n_steps, dtype, _plant_odd_frames if planted else None)
    return Workload(f"small_{gran}", F, H, W, C, heads, head_dim, n_ctx, dtype, gran, r, r_frame,
                    patch_k, steps, None if ctx is None else _store(ctx, dtype), *w)
