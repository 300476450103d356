"""Pre-bound calls for tight loops (benchmarks, serving): the ctypes argument
structures, workspace and output buffers are built once, so each call is a
single C-ABI call with no Python-side allocation."""
from __future__ import annotations

import ctypes as C
from typing import Dict, Optional

import torch

from . import _lib as L
from .api import Cfg, LayerCache, Shape, _need, _stream, _weights, workspace


class LayerRunner:
    """oc_layer_cached on a fixed shape, cfg, weights, cache and workspace."""

    def __init__(self, shape: Shape, cfg: Cfg, weights: Dict[str, torch.Tensor], device,
                 ctx: Optional[torch.Tensor] = None):
        self.shape, self.cfg = shape, cfg
        self._w = _weights(weights, shape)
        self.weights = weights
        self.cache = LayerCache(shape, device)
        self.ws = workspace(shape, cfg, device)
        self.ctx = ctx
        self.y_ctx = None
        if shape.n_ctx > 0:
            _need(ctx, shape.torch_dtype, "ctx")
            self.y_ctx = torch.empty((shape.n_ctx, shape.C), dtype=shape.torch_dtype, device=device)
        self._sh, self._cf = shape.c(), cfg.c()
        self._c = L.oc_cache(self.cache.y.data_ptr(), 0, 0)
        self._stream = _stream(self.cache.y)
        self._fn = L.lib().oc_layer_cached
        self._args_tail = (C.byref(self._w), C.byref(self._c), self.y_ctx.data_ptr() if self.y_ctx is not None else None,
                           None, self.ws.data_ptr(), self.ws.numel(), self._stream)
        self._ctx_ptr = ctx.data_ptr() if ctx is not None else None

    def reset(self):
        self._c.valid = 0
        self._c.step = 0

    def use_current_stream(self):
        """Launch on torch's current stream from now on (e.g. under graph capture)."""
        self._stream = _stream(self.cache.y)
        self._args_tail = self._args_tail[:-1] + (self._stream,)

    def __call__(self, x: torch.Tensor) -> torch.Tensor:
        st = self._fn(C.byref(self._sh), C.byref(self._cf), x.data_ptr(), self._ctx_ptr, *self._args_tail)
        if st != 0:
            L.check(st)
        self.cache.valid, self.cache.step = self._c.valid, self._c.step
        return self.cache.y


class FullRunner:
    """oc_attn_full (the uncached layer) on a fixed shape, weights and workspace."""

    def __init__(self, shape: Shape, cfg: Cfg, weights: Dict[str, torch.Tensor], device,
                 ctx: Optional[torch.Tensor] = None):
        self._w = _weights(weights, shape)
        self.weights = weights
        self.ws = workspace(shape, cfg, device)
        self.y = torch.empty((shape.F, shape.N, shape.C), dtype=shape.torch_dtype, device=device)
        self.y_ctx = None
        if shape.n_ctx > 0:
            self.y_ctx = torch.empty((shape.n_ctx, shape.C), dtype=shape.torch_dtype, device=device)
        self._sh, self._cf = shape.c(), cfg.c()
        self._fn = L.lib().oc_attn_full
        self._ctx_ptr = ctx.data_ptr() if ctx is not None else None
        self._tail = (C.byref(self._w), self.y.data_ptr(), self.y_ctx.data_ptr() if self.y_ctx is not None else None,
                      self.ws.data_ptr(), self.ws.numel(), _stream(self.y))

    def use_current_stream(self):
        """Launch on torch's current stream from now on (e.g. under graph capture)."""
        self._tail = self._tail[:-1] + (_stream(self.y),)

    def __call__(self, x: torch.Tensor) -> torch.Tensor:
        st = self._fn(C.byref(self._sh), C.byref(self._cf), x.data_ptr(), self._ctx_ptr, *self._tail)
        if st != 0:
            L.check(st)
        return self.y


class BlockRunner:
    """oc_block_cached (spatial layer with Frame / Token Cache, residual,
    temporal layer with Block Cache) on fixed shapes, weights and caches."""

    def __init__(self, shape: Shape, spatial: Cfg, temporal: Cfg, w_spatial: Dict[str, torch.Tensor],
                 w_temporal: Dict[str, torch.Tensor], device):
        from .api import block_workspace
        self._ws_, self._wt_ = _weights(w_spatial, shape), _weights(w_temporal, shape)
        self.weights = (w_spatial, w_temporal)
        self.cache_s, self.cache_t = LayerCache(shape, device), LayerCache(shape, device)
        self.h = torch.empty((shape.F, shape.N, shape.C), dtype=shape.torch_dtype, device=device)
        self.ws = block_workspace(shape, spatial, temporal, device)
        self._sh, self._cs, self._ct = shape.c(), spatial.c(), temporal.c()
        self._c_s = L.oc_cache(self.cache_s.y.data_ptr(), 0, 0)
        self._c_t = L.oc_cache(self.cache_t.y.data_ptr(), 0, 0)
        self._fn = L.lib().oc_block_cached
        self._tail = (C.byref(self._ws_), C.byref(self._wt_), C.byref(self._c_s), C.byref(self._c_t),
                      self.h.data_ptr(), None, None, self.ws.data_ptr(), self.ws.numel(), _stream(self.h))

    def reset(self):
        for c in (self._c_s, self._c_t):
            c.valid = 0
            c.step = 0

    def __call__(self, x: torch.Tensor) -> torch.Tensor:
        st = self._fn(C.byref(self._sh), C.byref(self._cs), C.byref(self._ct), x.data_ptr(), *self._tail)
        if st != 0:
            L.check(st)
        self.cache_s.valid, self.cache_s.step = self._c_s.valid, self._c_s.step
        self.cache_t.valid, self.cache_t.step = self._c_t.valid, self._c_t.step
        return self.cache_t.y


class FullBlockRunner:
    """The uncached block: full spatial attention, residual, full temporal
    attention (oc_attn_full, oc_residual_add, oc_attn_full)."""

    def __init__(self, shape: Shape, w_spatial: Dict[str, torch.Tensor], w_temporal: Dict[str, torch.Tensor],
                 device):
        self.spatial = FullRunner(shape, Cfg("token", 0.0), w_spatial, device)
        self.temporal = FullRunner(shape, Cfg("block", 0.0), w_temporal, device)
        self.h = torch.empty((shape.F, shape.N, shape.C), dtype=shape.torch_dtype, device=device)
        self._sh = shape.c()
        self._add = L.lib().oc_residual_add
        self._stream = _stream(self.h)

    def __call__(self, x: torch.Tensor) -> torch.Tensor:
        ys = self.spatial(x)
        st = self._add(C.byref(self._sh), x.data_ptr(), ys.data_ptr(), self.h.data_ptr(), self._stream)
        if st != 0:
            L.check(st)
        return self.temporal(self.h)


class FfnRunner:
    """oc_ffn_reduced on fixed weights: rows kept_idx (None: every token)
    written in place into y."""

    def __init__(self, shape: Shape, weights: Dict[str, torch.Tensor], kept_idx: Optional[torch.Tensor], device):
        from .api import ffn_workspace_bytes
        w1, w2 = weights["w1"], weights["w2"]
        self.hidden = w1.shape[0]
        self.kept = kept_idx
        self.n = kept_idx.numel() if kept_idx is not None else shape.F * shape.N
        self.y = torch.empty((shape.F, shape.N, shape.C), dtype=shape.torch_dtype, device=device)
        self.ws = torch.empty(max(ffn_workspace_bytes(shape, self.hidden, self.n), 256), dtype=torch.uint8,
                              device=device)
        self._fw = L.oc_ffn_weights(w1.data_ptr(), w2.data_ptr(), self.hidden, 0)
        self.weights = weights
        self._sh = shape.c()
        self._fn = L.lib().oc_ffn_reduced
        self._idx = kept_idx.data_ptr() if kept_idx is not None else None
        self._tail = (C.byref(self._fw), self.y.data_ptr(), 1, self.ws.data_ptr(), self.ws.numel(), _stream(self.y))

    def __call__(self, x: torch.Tensor) -> torch.Tensor:
        st = self._fn(C.byref(self._sh), x.data_ptr(), self._idx, self.n, *self._tail)
        if st != 0:
            L.check(st)
        return self.y
