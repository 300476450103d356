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
