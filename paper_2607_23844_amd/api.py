"""Python entry points with the same names as the C ABI (include/oc.h).

Argument marshalling only: torch supplies device memory and the current
stream; every step runs in the HIP library.  Tensors must be contiguous,
on the same GPU, bf16 or fp32 as the shape says; int tensors are int32.
"""
from __future__ import annotations

import ctypes as C
from dataclasses import dataclass
from typing import Dict, Optional, Tuple

import torch

from . import _lib as L


@dataclass(frozen=True)
class Shape:
    """Token tensor [F, N=H*W, C] of one attention layer plus its heads."""
    F: int
    H: int
    W: int
    C: int
    heads: int
    head_dim: int
    n_ctx: int = 0
    dtype: str = "bf16"      # "bf16" or "f32"

    @property
    def N(self) -> int:
        return self.H * self.W

    @property
    def torch_dtype(self) -> torch.dtype:
        return torch.bfloat16 if self.dtype == "bf16" else torch.float32

    def c(self) -> L.oc_shape:
        return L.oc_shape(self.F, self.H, self.W, self.C, self.heads, self.head_dim, self.n_ctx,
                          L.OC_BF16 if self.dtype == "bf16" else L.OC_F32)


@dataclass(frozen=True)
class Cfg:
    gran: str = "token"      # token | frame | block | frame_token
    r: float = 0.0
    r_frame: float = 0.0
    patch_k: int = 1
    cold: str = "matched"    # matched | full
    coarse_k: int = 0        # second, coarser level of the hierarchy (Token / Block Cache); 0: none
    r_coarse: float = 0.0

    def c(self) -> L.oc_cfg:
        return L.oc_cfg(L.GRANS[self.gran], self.patch_k, self.r, self.r_frame, L.COLDS[self.cold], self.coarse_k,
                        self.r_coarse)


@dataclass
class PlanInfo:
    n_groups: int
    n_src_max: int
    n_dst_max: int
    n_frame_src: int
    n_frame_dst: int
    n_frame_cached: int
    n_kept: int
    n_cached: int
    n_seq: int
    seq_len: int
    workspace_bytes: int


class LayerCache:
    """The layer cache of one attention layer: a device buffer [F, N, C] that
    is also the layer output, plus the host-side valid flag and step count."""

    def __init__(self, shape: Shape, device, y: Optional[torch.Tensor] = None):
        self.shape = shape
        self.y = y if y is not None else torch.empty((shape.F, shape.N, shape.C), dtype=shape.torch_dtype,
                                                     device=device)
        self.valid = 0
        self.step = 0


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(t: torch.Tensor) -> int:
    return torch.cuda.current_stream(t.device).cuda_stream


def _need(t: torch.Tensor, dtype: torch.dtype, name: str) -> None:
    if not t.is_cuda:
        raise L.OmniCacheError(L.OC_ERR_INVALID_ARG, f"{name} must be a GPU tensor")
    if t.dtype != dtype:
        raise L.OmniCacheError(L.OC_ERR_DTYPE, f"{name} has dtype {t.dtype}, expected {dtype}")
    if not t.is_contiguous():
        raise L.OmniCacheError(L.OC_ERR_INVALID_ARG, f"{name} must be contiguous")


def _weights(w: Dict[str, torch.Tensor], shape: Shape) -> L.oc_attn_weights:
    hd = shape.heads * shape.head_dim
    for k, s in (("wq", (hd, shape.C)), ("wk", (hd, shape.C)), ("wv", (hd, shape.C)), ("wo", (shape.C, hd))):
        _need(w[k], shape.torch_dtype, k)
        if tuple(w[k].shape) != s:
            raise L.OmniCacheError(L.OC_ERR_SHAPE, f"{k} has shape {tuple(w[k].shape)}, expected {s}")
    return L.oc_attn_weights(w["wq"].data_ptr(), w["wk"].data_ptr(), w["wv"].data_ptr(), w["wo"].data_ptr())


def plan(shape: Shape, cfg: Cfg) -> PlanInfo:
    info = L.oc_plan_info()
    sh, cf = shape.c(), cfg.c()
    L.check(L.lib().oc_plan(C.byref(sh), C.byref(cf), C.byref(info)))
    return PlanInfo(*(getattr(info, f) for f, _ in L.oc_plan_info._fields_))


def workspace(shape: Shape, cfg: Cfg, device) -> torch.Tensor:
    return torch.empty(max(plan(shape, cfg).workspace_bytes, 256), dtype=torch.uint8, device=device)


def match(x: torch.Tensor, shape: Shape, cfg: Cfg, ws: torch.Tensor, frames: bool = False):
    """(node_max [G, S] f32, node_idx [G, S] i32[, frame info dict])"""
    _need(x, shape.torch_dtype, "x")
    pl = plan(shape, cfg)
    dev = x.device
    nm = torch.empty((pl.n_groups, pl.n_src_max), dtype=torch.float32, device=dev)
    ni = torch.empty((pl.n_groups, pl.n_src_max), dtype=torch.int32, device=dev)
    fi = None
    out = {}
    if frames:
        out = dict(frame_max=torch.empty(max(pl.n_frame_src, 1), dtype=torch.float32, device=dev),
                   frame_idx=torch.empty(max(pl.n_frame_src, 1), dtype=torch.int32, device=dev),
                   pairs=torch.empty((max(pl.n_frame_cached, 1), 2), dtype=torch.int32, device=dev))
        fi = L.oc_frame_info(out["frame_max"].data_ptr(), out["frame_idx"].data_ptr(), out["pairs"].data_ptr())
    sh, cf = shape.c(), cfg.c()
    L.check(L.lib().oc_match(C.byref(sh), C.byref(cf), x.data_ptr(), nm.data_ptr(), ni.data_ptr(),
                             C.byref(fi) if fi is not None else None, ws.data_ptr(), ws.numel(), _stream(x)))
    if frames:
        out["frame_max"] = out["frame_max"][:pl.n_frame_src]
        out["frame_idx"] = out["frame_idx"][:pl.n_frame_src]
        out["pairs"] = out["pairs"][:pl.n_frame_cached]
        return nm, ni, out
    return nm, ni


def select(node_max: torch.Tensor, node_idx: torch.Tensor, shape: Shape, cfg: Cfg, ws: torch.Tensor,
           map_matched: bool = False) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor]:
    """(kept_idx [n_kept], cached_idx [n_cached], restore_map [F*N]), int32"""
    _need(node_max, torch.float32, "node_max")
    _need(node_idx, torch.int32, "node_idx")
    pl = plan(shape, cfg)
    dev = node_max.device
    kept = torch.empty(max(pl.n_kept, 1), dtype=torch.int32, device=dev)
    cached = torch.empty(max(pl.n_cached, 1), dtype=torch.int32, device=dev)
    rmap = torch.empty(shape.F * shape.N, dtype=torch.int32, device=dev)
    sh, cf = shape.c(), cfg.c()
    L.check(L.lib().oc_select(C.byref(sh), C.byref(cf), node_max.data_ptr(), node_idx.data_ptr(), kept.data_ptr(),
                              cached.data_ptr(), rmap.data_ptr(), 1 if map_matched else 0, ws.data_ptr(),
                              ws.numel(), _stream(node_max)))
    return kept[:pl.n_kept], cached[:pl.n_cached], rmap


def gather(x: torch.Tensor, kept_idx: torch.Tensor, shape: Shape, cfg: Cfg) -> torch.Tensor:
    _need(x, shape.torch_dtype, "x")
    _need(kept_idx, torch.int32, "kept_idx")
    pl = plan(shape, cfg)
    packed = cfg.gran == "frame" and cfg.patch_k > 1      # sequences of varying length: [n_kept, C]
    shp = (max(pl.n_kept, 1), shape.C) if packed else (max(pl.n_seq, 1), max(pl.seq_len, 1), shape.C)
    out = torch.empty(shp, dtype=x.dtype, device=x.device)
    sh, cf = shape.c(), cfg.c()
    L.check(L.lib().oc_gather(C.byref(sh), C.byref(cf), x.data_ptr(), kept_idx.data_ptr(), out.data_ptr(),
                              _stream(x)))
    return out[:pl.n_kept] if packed else out[:pl.n_seq, :pl.seq_len]


def attn_workspace_bytes(shape: Shape, n_seq: int, seq_len: int) -> int:
    sh = shape.c()
    return int(L.lib().oc_attn_workspace_bytes(C.byref(sh), n_seq, seq_len))


def attn_reduced(x_kept: torch.Tensor, n_seq: int, seq_len: int, weights: Dict[str, torch.Tensor], shape: Shape,
                 ctx: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None):
    """(y_kept [n_seq*seq_len, C], y_ctx [n_ctx, C] or None)"""
    _need(x_kept, shape.torch_dtype, "x_kept")
    w = _weights(weights, shape)
    dev = x_kept.device
    y = torch.empty((max(n_seq * seq_len, 1), shape.C), dtype=x_kept.dtype, device=dev)
    y_ctx = None
    if shape.n_ctx > 0:
        _need(ctx, shape.torch_dtype, "ctx")
        y_ctx = torch.empty((shape.n_ctx, shape.C), dtype=x_kept.dtype, device=dev)
    need = attn_workspace_bytes(shape, n_seq, seq_len)
    if ws is None:
        ws = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
    sh = shape.c()
    L.check(L.lib().oc_attn_reduced(C.byref(sh), x_kept.data_ptr(), n_seq, seq_len, _ptr(ctx), C.byref(w),
                                    y.data_ptr(), _ptr(y_ctx), ws.data_ptr(), ws.numel(), _stream(x_kept)))
    return y[:n_seq * seq_len], y_ctx


def restore(y_kept: torch.Tensor, restore_map: torch.Tensor, shape: Shape, cache_y: Optional[torch.Tensor] = None,
            y: Optional[torch.Tensor] = None) -> torch.Tensor:
    _need(y_kept, shape.torch_dtype, "y_kept")
    _need(restore_map, torch.int32, "restore_map")
    if y is None:
        y = torch.empty((shape.F, shape.N, shape.C), dtype=y_kept.dtype, device=y_kept.device)
    sh = shape.c()
    L.check(L.lib().oc_restore(C.byref(sh), y_kept.data_ptr(), y_kept.shape[0], restore_map.data_ptr(),
                               _ptr(cache_y), y.data_ptr(), _stream(y_kept)))
    return y


def _trace(shape: Shape, cfg: Cfg, cache: LayerCache, pl: PlanInfo, dev):
    """Device buffers for a layer call's decisions and the oc_trace pointing
    at them (a cold "full" step runs with every ratio at 0)."""
    cold_full = cache.valid == 0 and cfg.cold == "full"
    tp = plan(shape, Cfg(cfg.gran, 0.0, 0.0, cfg.patch_k, cfg.cold, cfg.coarse_k, 0.0)) if cold_full else pl
    n_kept, n_cached = tp.n_kept, tp.n_cached
    out = dict(node_max=torch.empty((tp.n_groups, tp.n_src_max), dtype=torch.float32, device=dev),
               node_idx=torch.empty((tp.n_groups, tp.n_src_max), dtype=torch.int32, device=dev),
               kept_idx=torch.empty(max(n_kept, 1), dtype=torch.int32, device=dev),
               cached_idx=torch.empty(max(n_cached, 1), dtype=torch.int32, device=dev),
               restore_map=torch.empty(shape.F * shape.N, dtype=torch.int32, device=dev),
               frame_max=torch.empty(max(pl.n_frame_src, 1), dtype=torch.float32, device=dev),
               frame_idx=torch.empty(max(pl.n_frame_src, 1), dtype=torch.int32, device=dev),
               pairs=torch.empty((max(pl.n_frame_cached, 1), 2), dtype=torch.int32, device=dev))
    fi = L.oc_frame_info(out["frame_max"].data_ptr(), out["frame_idx"].data_ptr(), out["pairs"].data_ptr())
    tr = L.oc_trace(out["node_max"].data_ptr(), out["node_idx"].data_ptr(), out["kept_idx"].data_ptr(),
                    out["cached_idx"].data_ptr(), out["restore_map"].data_ptr(), fi)
    out["kept_idx"] = out["kept_idx"][:n_kept]
    out["cached_idx"] = out["cached_idx"][:n_cached]
    out["frame_max"] = out["frame_max"][:pl.n_frame_src]
    out["frame_idx"] = out["frame_idx"][:pl.n_frame_src]
    out["pairs"] = out["pairs"][:tp.n_frame_cached]
    return tr, out


def _layer_args(x, weights, cache, shape, cfg, ctx, trace):
    _need(x, shape.torch_dtype, "x")
    _need(cache.y, shape.torch_dtype, "cache.y")
    w = _weights(weights, shape)
    dev = x.device
    pl = plan(shape, cfg)
    y_ctx = None
    if shape.n_ctx > 0:
        _need(ctx, shape.torch_dtype, "ctx")
        y_ctx = torch.empty((shape.n_ctx, shape.C), dtype=x.dtype, device=dev)
    tr, out = _trace(shape, cfg, cache, pl, dev) if trace else (None, None)
    c = L.oc_cache(cache.y.data_ptr(), cache.valid, cache.step)
    return w, pl, y_ctx, tr, out, c


def layer_cached(x: torch.Tensor, weights: Dict[str, torch.Tensor], cache: LayerCache, shape: Shape, cfg: Cfg,
                 ctx: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None, trace: bool = False):
    """One cached layer call; returns (cache.y, y_ctx, trace dict or None)."""
    w, pl, y_ctx, tr, out, c = _layer_args(x, weights, cache, shape, cfg, ctx, trace)
    if ws is None:
        ws = workspace(shape, cfg, x.device)
    sh, cf = shape.c(), cfg.c()
    L.check(L.lib().oc_layer_cached(C.byref(sh), C.byref(cf), x.data_ptr(), _ptr(ctx), C.byref(w), C.byref(c),
                                    _ptr(y_ctx), C.byref(tr) if tr is not None else None, ws.data_ptr(), ws.numel(),
                                    _stream(x)))
    cache.valid, cache.step = c.valid, c.step
    return cache.y, y_ctx, out


def layer_cached_static(x: torch.Tensor, weights: Dict[str, torch.Tensor], cache: LayerCache, shape: Shape,
                        cfg: Cfg, ctx: Optional[torch.Tensor] = None, trace: bool = False):
    """oc_layer_cached_static: the same layer call with the library's own
    device scratch instead of a workspace (the library allocates nothing;
    the binding allocates only the outputs it returns: y_ctx and the trace
    buffers when asked for)."""
    w, pl, y_ctx, tr, out, c = _layer_args(x, weights, cache, shape, cfg, ctx, trace)
    sh, cf = shape.c(), cfg.c()
    L.check(L.lib().oc_layer_cached_static(C.byref(sh), C.byref(cf), x.data_ptr(), _ptr(ctx), C.byref(w),
                                           C.byref(c), _ptr(y_ctx), C.byref(tr) if tr is not None else None,
                                           _stream(x)))
    cache.valid, cache.step = c.valid, c.step
    return cache.y, y_ctx, out


def ffn_workspace_bytes(shape: Shape, hidden: int, n_rows: int) -> int:
    sh = shape.c()
    return int(L.lib().oc_ffn_workspace_bytes(C.byref(sh), hidden, n_rows))


def ffn_reduced(x: torch.Tensor, weights: Dict[str, torch.Tensor], shape: Shape,
                kept_idx: Optional[torch.Tensor] = None, n_rows: Optional[int] = None,
                y: Optional[torch.Tensor] = None, scatter: bool = True,
                ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """oc_ffn_reduced: GELU(x[t] W1^T) W2^T for the retained tokens t of
    kept_idx (all tokens when None).  scatter: written into y [F, N, C] at
    their positions (other rows untouched); else y is [n_rows, C]."""
    _need(x, shape.torch_dtype, "x")
    w1, w2 = weights["w1"], weights["w2"]
    hidden = w1.shape[0]
    for k, t, s in (("w1", w1, (hidden, shape.C)), ("w2", w2, (shape.C, hidden))):
        _need(t, shape.torch_dtype, k)
        if tuple(t.shape) != s:
            raise L.OmniCacheError(L.OC_ERR_SHAPE, f"{k} has shape {tuple(t.shape)}, expected {s}")
    if kept_idx is not None:
        _need(kept_idx, torch.int32, "kept_idx")
        n = kept_idx.numel() if n_rows is None else n_rows
    else:
        n = shape.F * shape.N if n_rows is None else n_rows
    dev = x.device
    if y is None:
        y = torch.empty((shape.F, shape.N, shape.C) if scatter else (max(n, 1), shape.C), dtype=x.dtype, device=dev)
    _need(y, shape.torch_dtype, "y")
    if ws is None:
        ws = torch.empty(max(ffn_workspace_bytes(shape, hidden, n), 256), dtype=torch.uint8, device=dev)
    fw = L.oc_ffn_weights(w1.data_ptr(), w2.data_ptr(), hidden, 0)
    sh = shape.c()
    L.check(L.lib().oc_ffn_reduced(C.byref(sh), x.data_ptr(), _ptr(kept_idx), n, C.byref(fw), y.data_ptr(),
                                   1 if scatter else 0, ws.data_ptr(), ws.numel(), _stream(x)))
    return y if scatter else y[:n]


def layered_schedule(latency, quality, target_speedup: float, interval: int, mask=None):
    """oc_layered_schedule (§3.4, Alg. 1) on host tables [n_layers, n_steps]:
    returns ([(layer, step, interval), ...] in selection order, saved, budget)."""
    import numpy as np
    lat = np.ascontiguousarray(latency, dtype=np.float64)
    qual = np.ascontiguousarray(quality, dtype=np.float64)
    if lat.ndim != 2 or qual.shape != lat.shape:
        raise L.OmniCacheError(L.OC_ERR_SHAPE, "latency and quality must be equal-shaped 2-D tables")
    m = None if mask is None else np.ascontiguousarray(mask, dtype=np.uint8)
    if m is not None and m.shape != lat.shape:
        raise L.OmniCacheError(L.OC_ERR_SHAPE, "mask must have the tables' shape")
    n_l, n_t = lat.shape
    cap = max(n_l * n_t, 1)
    out = (L.oc_cache_entry * cap)()
    n, saved, budget = C.c_int32(), C.c_double(), C.c_double()
    L.check(L.lib().oc_layered_schedule(n_l, n_t, lat.ctypes.data, qual.ctypes.data,
                                        None if m is None else m.ctypes.data, float(target_speedup), int(interval),
                                        out, cap, C.byref(n), C.byref(saved), C.byref(budget)))
    return [(out[i].layer, out[i].step, out[i].interval) for i in range(n.value)], saved.value, budget.value


def residual_add(x: torch.Tensor, y: torch.Tensor, shape: Shape, h: Optional[torch.Tensor] = None) -> torch.Tensor:
    """oc_residual_add: h = x + y over [F, N, C]."""
    _need(x, shape.torch_dtype, "x")
    _need(y, shape.torch_dtype, "y")
    if h is None:
        h = torch.empty_like(x)
    _need(h, shape.torch_dtype, "h")
    sh = shape.c()
    L.check(L.lib().oc_residual_add(C.byref(sh), x.data_ptr(), y.data_ptr(), h.data_ptr(), _stream(x)))
    return h


def block_workspace(shape: Shape, spatial: Cfg, temporal: Cfg, device) -> torch.Tensor:
    sh, cs, ct = shape.c(), spatial.c(), temporal.c()
    n = int(L.lib().oc_block_workspace_bytes(C.byref(sh), C.byref(cs), C.byref(ct)))
    return torch.empty(max(n, 256), dtype=torch.uint8, device=device)


def block_cached(x: torch.Tensor, w_spatial: Dict[str, torch.Tensor], w_temporal: Dict[str, torch.Tensor],
                 cache_spatial: LayerCache, cache_temporal: LayerCache, shape: Shape, spatial: Cfg, temporal: Cfg,
                 h: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None, trace: bool = False):
    """oc_block_cached: the spatial layer (Frame / Token Cache), the residual
    h = x + y_spatial and the temporal layer (Block Cache) in one call.
    Returns (cache_temporal.y, h, spatial trace, temporal trace)."""
    wsc, _, _, tr_s, out_s, c_s = _layer_args(x, w_spatial, cache_spatial, shape, spatial, None, trace)
    wtc, _, _, tr_t, out_t, c_t = _layer_args(x, w_temporal, cache_temporal, shape, temporal, None, trace)
    if h is None:
        h = torch.empty_like(x)
    _need(h, shape.torch_dtype, "h")
    if ws is None:
        ws = block_workspace(shape, spatial, temporal, x.device)
    sh, cs, ct = shape.c(), spatial.c(), temporal.c()
    L.check(L.lib().oc_block_cached(C.byref(sh), C.byref(cs), C.byref(ct), x.data_ptr(), C.byref(wsc), C.byref(wtc),
                                    C.byref(c_s), C.byref(c_t), h.data_ptr(),
                                    C.byref(tr_s) if tr_s is not None else None,
                                    C.byref(tr_t) if tr_t is not None else None, ws.data_ptr(), ws.numel(),
                                    _stream(x)))
    cache_spatial.valid, cache_spatial.step = c_s.valid, c_s.step
    cache_temporal.valid, cache_temporal.step = c_t.valid, c_t.step
    return cache_temporal.y, h, out_s, out_t


def static_scratch_bytes() -> int:
    return int(L.lib().oc_static_scratch_bytes())


def attn_full(x: torch.Tensor, weights: Dict[str, torch.Tensor], shape: Shape, cfg: Cfg,
              ctx: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None):
    """The uncached layer on the same input: (y [F, N, C], y_ctx)."""
    _need(x, shape.torch_dtype, "x")
    w = _weights(weights, shape)
    dev = x.device
    if ws is None:
        ws = workspace(shape, cfg, dev)
    y = torch.empty((shape.F, shape.N, shape.C), dtype=x.dtype, device=dev)
    y_ctx = None
    if shape.n_ctx > 0:
        _need(ctx, shape.torch_dtype, "ctx")
        y_ctx = torch.empty((shape.n_ctx, shape.C), dtype=x.dtype, device=dev)
    sh, cf = shape.c(), cfg.c()
    L.check(L.lib().oc_attn_full(C.byref(sh), C.byref(cf), x.data_ptr(), _ptr(ctx), C.byref(w), y.data_ptr(),
                                 _ptr(y_ctx), ws.data_ptr(), ws.numel(), _stream(x)))
    return y, y_ctx


class StageTimer:
    """Per-stage kernel time while this timer is attached to the calling
    thread: every library kernel is launched with a pair of the timer's HIP
    events, stamped by the runtime at the kernel's start and end."""

    def __init__(self):
        self._t = C.c_void_p()
        L.check(L.lib().oc_timer_create(C.byref(self._t)))

    def __enter__(self):
        L.check(L.lib().oc_timer_use(self._t))
        return self

    def __exit__(self, *exc):
        L.lib().oc_timer_use(None)
        return False

    def reset(self):
        L.check(L.lib().oc_timer_reset(self._t))

    def collect(self) -> Dict[str, Tuple[float, int]]:
        """{stage: (total ms, launches)} including everything recorded so far."""
        L.check(L.lib().oc_timer_collect(self._t))
        out = {}
        for i in range(L.lib().oc_timer_stage_count(self._t)):
            name, ms, n = C.c_char_p(), C.c_double(), C.c_int64()
            L.check(L.lib().oc_timer_stage(self._t, i, C.byref(name), C.byref(ms), C.byref(n)))
            out[name.value.decode()] = (ms.value, n.value)
        return out

    def __del__(self):
        try:
            if self._t:
                L.lib().oc_timer_destroy(self._t)
        except Exception:
            pass


def clock_sample(samples: torch.Tensor, n: int, gap_ticks: int, stream: Optional[torch.cuda.Stream] = None) -> None:
    """Enqueue the shader clock sampler (oc_clock_sample) on `stream` (the
    current stream if None): n pairs (shader clock, 100 MHz real-time clock)
    into the int64 device tensor `samples` of at least 2n elements."""
    _need(samples, torch.int64, "samples")
    if samples.numel() < 2 * n:
        raise ValueError("samples must hold 2n int64 values")
    st = stream.cuda_stream if stream is not None else _stream(samples)
    L.check(L.lib().oc_clock_sample(samples.data_ptr(), n, gap_ticks, st))


def clock_ghz(samples: torch.Tensor) -> "np.ndarray":
    """Shader clock in GHz over each interval of a finished clock_sample."""
    import numpy as np
    a = samples.view(-1, 2).cpu().numpy().astype(np.float64)
    return np.diff(a[:, 0]) / (np.diff(a[:, 1]) * 10.0)
