"""ctypes view of include/oc.h.  Loads the in-tree liboc.so (or the build
that OC_LIBRARY names, such as the host-sanitized liboc_asan.so) and fails
loudly if it has not been built: there is no fallback implementation."""
from __future__ import annotations

import ctypes as C
import os

LIB_PATH = os.environ.get("OC_LIBRARY") or os.path.join(os.path.dirname(os.path.abspath(__file__)), "liboc.so")

OC_OK, OC_ERR_INVALID_ARG, OC_ERR_SHAPE, OC_ERR_DTYPE, OC_ERR_WORKSPACE, OC_ERR_CACHE_STATE, OC_ERR_HIP = range(7)
OC_F32, OC_BF16 = 0, 1
GRANS = {"token": 0, "frame": 1, "block": 2, "frame_token": 3}
COLDS = {"matched": 0, "full": 1}


class OmniCacheError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{_STATUS_NAMES.get(status, status)}: {message}")
        self.status = status
        self.message = message


_STATUS_NAMES = {0: "OC_OK", 1: "OC_ERR_INVALID_ARG", 2: "OC_ERR_SHAPE", 3: "OC_ERR_DTYPE",
                 4: "OC_ERR_WORKSPACE", 5: "OC_ERR_CACHE_STATE", 6: "OC_ERR_HIP"}


class oc_shape(C.Structure):
    _fields_ = [("F", C.c_int32), ("H", C.c_int32), ("W", C.c_int32), ("C", C.c_int32),
                ("heads", C.c_int32), ("head_dim", C.c_int32), ("n_ctx", C.c_int32), ("dtype", C.c_int32)]


class oc_cfg(C.Structure):
    _fields_ = [("gran", C.c_int32), ("patch_k", C.c_int32), ("r", C.c_double), ("r_frame", C.c_double),
                ("cold", C.c_int32), ("coarse_k", C.c_int32), ("r_coarse", C.c_double)]


class oc_cache(C.Structure):
    _fields_ = [("y", C.c_void_p), ("valid", C.c_int32), ("step", C.c_int32)]


class oc_attn_weights(C.Structure):
    _fields_ = [("wq", C.c_void_p), ("wk", C.c_void_p), ("wv", C.c_void_p), ("wo", C.c_void_p)]


class oc_plan_info(C.Structure):
    _fields_ = [("n_groups", C.c_int32), ("n_src_max", C.c_int32), ("n_dst_max", C.c_int32),
                ("n_frame_src", C.c_int32), ("n_frame_dst", C.c_int32), ("n_frame_cached", C.c_int32),
                ("n_kept", C.c_int32), ("n_cached", C.c_int32), ("n_seq", C.c_int32), ("seq_len", C.c_int32),
                ("workspace_bytes", C.c_size_t)]


class oc_ffn_weights(C.Structure):
    _fields_ = [("w1", C.c_void_p), ("w2", C.c_void_p), ("hidden", C.c_int32), ("reserved", C.c_int32)]


class oc_cache_entry(C.Structure):
    _fields_ = [("layer", C.c_int32), ("step", C.c_int32), ("interval", C.c_int32)]


class oc_frame_info(C.Structure):
    _fields_ = [("frame_max", C.c_void_p), ("frame_idx", C.c_void_p), ("pairs", C.c_void_p)]


class oc_trace(C.Structure):
    _fields_ = [("node_max", C.c_void_p), ("node_idx", C.c_void_p), ("kept_idx", C.c_void_p),
                ("cached_idx", C.c_void_p), ("restore_map", C.c_void_p), ("frames", oc_frame_info)]


P = C.POINTER
_SIGS = {
    "oc_plan": (C.c_int, [P(oc_shape), P(oc_cfg), P(oc_plan_info)]),
    "oc_match": (C.c_int, [P(oc_shape), P(oc_cfg), C.c_void_p, C.c_void_p, C.c_void_p, P(oc_frame_info),
                           C.c_void_p, C.c_size_t, C.c_void_p]),
    "oc_select": (C.c_int, [P(oc_shape), P(oc_cfg), C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                            C.c_int32, C.c_void_p, C.c_size_t, C.c_void_p]),
    "oc_gather": (C.c_int, [P(oc_shape), P(oc_cfg), C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]),
    "oc_attn_reduced": (C.c_int, [P(oc_shape), C.c_void_p, C.c_int32, C.c_int32, C.c_void_p, P(oc_attn_weights),
                                  C.c_void_p, C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]),
    "oc_attn_workspace_bytes": (C.c_size_t, [P(oc_shape), C.c_int32, C.c_int32]),
    "oc_restore": (C.c_int, [P(oc_shape), C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]),
    "oc_layer_cached": (C.c_int, [P(oc_shape), P(oc_cfg), C.c_void_p, C.c_void_p, P(oc_attn_weights), P(oc_cache),
                                  C.c_void_p, P(oc_trace), C.c_void_p, C.c_size_t, C.c_void_p]),
    "oc_ffn_reduced": (C.c_int, [P(oc_shape), C.c_void_p, C.c_void_p, C.c_int32, P(oc_ffn_weights), C.c_void_p,
                                 C.c_int32, C.c_void_p, C.c_size_t, C.c_void_p]),
    "oc_ffn_workspace_bytes": (C.c_size_t, [P(oc_shape), C.c_int32, C.c_int32]),
    "oc_layered_schedule": (C.c_int, [C.c_int32, C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p, C.c_double,
                                      C.c_int32, P(oc_cache_entry), C.c_int32, P(C.c_int32), P(C.c_double),
                                      P(C.c_double)]),
    "oc_residual_add": (C.c_int, [P(oc_shape), C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]),
    "oc_block_cached": (C.c_int, [P(oc_shape), P(oc_cfg), P(oc_cfg), C.c_void_p, P(oc_attn_weights),
                                  P(oc_attn_weights), P(oc_cache), P(oc_cache), C.c_void_p, P(oc_trace), P(oc_trace),
                                  C.c_void_p, C.c_size_t, C.c_void_p]),
    "oc_block_workspace_bytes": (C.c_size_t, [P(oc_shape), P(oc_cfg), P(oc_cfg)]),
    "oc_layer_cached_static": (C.c_int, [P(oc_shape), P(oc_cfg), C.c_void_p, C.c_void_p, P(oc_attn_weights),
                                         P(oc_cache), C.c_void_p, P(oc_trace), C.c_void_p]),
    "oc_static_scratch_bytes": (C.c_size_t, []),
    "oc_attn_full": (C.c_int, [P(oc_shape), P(oc_cfg), C.c_void_p, C.c_void_p, P(oc_attn_weights), C.c_void_p,
                               C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]),
    "oc_status_string": (C.c_char_p, [C.c_int]),
    "oc_last_error": (C.c_char_p, []),
    "oc_timer_create": (C.c_int, [P(C.c_void_p)]),
    "oc_timer_destroy": (None, [C.c_void_p]),
    "oc_timer_use": (C.c_int, [C.c_void_p]),
    "oc_timer_collect": (C.c_int, [C.c_void_p]),
    "oc_timer_reset": (C.c_int, [C.c_void_p]),
    "oc_timer_stage_count": (C.c_int32, [C.c_void_p]),
    "oc_timer_stage": (C.c_int, [C.c_void_p, C.c_int32, P(C.c_char_p), P(C.c_double), P(C.c_int64)]),
    "oc_clock_sample": (C.c_int, [C.c_void_p, C.c_int32, C.c_int32, C.c_void_p]),
}

_lib = None


def lib() -> C.CDLL:
    """The loaded library; raises if it is missing (build it first)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise OmniCacheError(OC_ERR_HIP, f"{LIB_PATH} is not built: run `python -m paper_2607_23844_amd.build`")
        L = C.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def check(status: int) -> None:
    if status != OC_OK:
        raise OmniCacheError(status, lib().oc_last_error().decode())
