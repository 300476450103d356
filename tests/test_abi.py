"""The C-ABI library: it loads, exports every symbol include/oc.h declares,
plans static sizes that agree with the oracle's group and sequence counts,
and rejects bad arguments on the host before launching anything.  No test
here touches a GPU."""
import ctypes as C
import os
import re

import numpy as np
import pytest

import paper_2607_23844_amd as oc
from paper_2607_23844_amd import _lib as L
from oracle import oc_oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "oc.h")


@pytest.fixture(scope="module", autouse=True)
def built():
    if not os.path.exists(L.LIB_PATH):
        from paper_2607_23844_amd import build
        build.build()
    return L.lib()


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:oc_status|size_t|const char \*|void|int32_t)\s*(oc_\w+)\s*\(", text,
                                 re.M)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("oc_match", "oc_select", "oc_gather", "oc_attn_reduced", "oc_restore", "oc_layer_cached",
                     "oc_plan", "oc_attn_full"):
        assert required in names


def test_library_exports_every_declared_symbol():
    lib = C.CDLL(L.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_library_leaves_no_library_symbol_undefined():
    """Every kernel and function of the library is defined in it: a kernel
    whose host stub the compiler dropped would only fail at its first launch
    (the library is loaded with lazy binding)."""
    import shutil
    import subprocess
    nm = shutil.which("nm")
    if nm is None:
        pytest.skip("nm not available")
    out = subprocess.run([nm, "-C", "--undefined-only", L.LIB_PATH], capture_output=True, text=True, check=True).stdout
    missing = [l.strip() for l in out.splitlines() if "oc::" in l or " oc_" in l]
    assert not missing, "undefined in the library: " + "; ".join(missing[:5])


def test_python_binding_covers_every_declared_symbol():
    assert set(declared_functions()) <= set(L._SIGS)


def test_struct_sizes_match_the_header_layout():
    assert C.sizeof(L.oc_shape) == 32
    assert C.sizeof(L.oc_cfg) == 40
    assert C.sizeof(L.oc_cache) == 16
    assert C.sizeof(L.oc_attn_weights) == 32
    assert C.sizeof(L.oc_plan_info) == 48
    assert C.sizeof(L.oc_trace) == 64
    assert C.sizeof(L.oc_ffn_weights) == 24
    assert C.sizeof(L.oc_cache_entry) == 12


WORKLOAD_SHAPES = [
    # name, shape, cfg
    ("tok16_f32", oc.Shape(1, 16, 16, 64, 1, 64, 0, "f32"), oc.Cfg("token", r=0.5)),
    ("sd3_1024_r25", oc.Shape(1, 64, 64, 1536, 24, 64, 333), oc.Cfg("token", r=0.25)),
    ("sd3_1024_r50", oc.Shape(1, 64, 64, 1536, 24, 64, 333), oc.Cfg("token", r=0.5)),
    ("sd3_1024_r75", oc.Shape(1, 64, 64, 1536, 24, 64, 333), oc.Cfg("token", r=0.75)),
    ("sd3_1024_k2", oc.Shape(1, 64, 64, 1536, 24, 64, 333), oc.Cfg("token", r=0.5, patch_k=2)),
    ("sd3_1024_k8", oc.Shape(1, 64, 64, 1536, 24, 64, 333), oc.Cfg("token", r=0.5, patch_k=8)),
    ("latte_spatial", oc.Shape(16, 16, 16, 1152, 16, 72), oc.Cfg("frame", r_frame=0.25)),
    ("latte_temporal", oc.Shape(16, 16, 16, 1152, 16, 72), oc.Cfg("block", r=0.5)),
    ("svdxt_level", oc.Shape(25, 72, 128, 320, 5, 64), oc.Cfg("frame_token", r=0.5, r_frame=0.2)),
    ("svdxt_level_k4", oc.Shape(25, 72, 128, 320, 5, 64), oc.Cfg("frame_token", r=0.5, r_frame=0.2, patch_k=4)),
    ("latte_spatial_k2", oc.Shape(16, 16, 16, 1152, 16, 72), oc.Cfg("frame", r_frame=0.25, patch_k=2)),
    ("latte_spatial_k4", oc.Shape(16, 16, 16, 1152, 16, 72), oc.Cfg("frame", r_frame=0.25, patch_k=4)),
]


def _oracle_counts(shape, cfg):
    """Group and sequence counts from the oracle's own group builders (no
    data needed: counts do not depend on which frames are paired)."""
    s = O.LayerShape(shape.F, shape.H, shape.W, shape.C, shape.heads, shape.head_dim, shape.n_ctx)
    k = cfg.patch_k
    if cfg.gran == "token":
        gs = O.token_groups(s, k, range(s.F), cfg.r)
        seq_len = s.N - sum(g.R for g in gs[:k * k])
        return len(gs), max(len(g.src) for g in gs), max(len(g.dst) for g in gs), s.F, seq_len
    if cfg.gran == "block":
        gs = O.block_groups(s, k, cfg.r)
        return len(gs), len(gs[0].src), len(gs[0].dst), s.N - sum(g.R for g in gs), s.F
    if cfg.gran == "frame" and k > 1:
        # per-patch frame groups; F sequences of at most N tokens
        gs = O.frame_patch_groups(s, k, cfg.r_frame)
        return len(gs), len(gs[0].src), len(gs[0].dst), s.F, s.N
    if cfg.gran == "frame":
        g = O.frame_group(s, cfg.r_frame)
        return 1, len(g.src), len(g.dst), s.F - g.R, s.N
    g = O.frame_group(s, cfg.r_frame)
    pairs = [(2 * i + 1, 2 * i) for i in range(g.R)]
    units = O._units(s, pairs)
    groups = []
    for u in units:
        groups += O.pair_token_groups(s, k, u[0], u[1], cfg.r) if len(u) == 2 else O.token_groups(s, k, [u[0]], cfg.r)
    per_unit = len(groups) // len(units)
    seq_len = 2 * s.N - sum(g.R for g in groups[:per_unit]) if len(units[0]) == 2 else \
        s.N - sum(g.R for g in groups[:per_unit])
    return len(groups), max(len(x.src) for x in groups), max(len(x.dst) for x in groups), len(units), seq_len


@pytest.mark.parametrize("name,shape,cfg", WORKLOAD_SHAPES, ids=[w[0] for w in WORKLOAD_SHAPES])
def test_plan_agrees_with_oracle_counts(name, shape, cfg):
    pl = oc.plan(shape, cfg)
    G, S, D, n_seq, seq_len = _oracle_counts(shape, cfg)
    assert (pl.n_groups, pl.n_src_max, pl.n_dst_max) == (G, S, D)
    assert (pl.n_seq, pl.seq_len) == (n_seq, seq_len)
    assert pl.n_kept + pl.n_cached == shape.F * shape.N
    assert pl.workspace_bytes > 0


def test_plan_known_sizes():
    pl = oc.plan(oc.Shape(1, 64, 64, 1536, 24, 64, 333), oc.Cfg("token", r=0.5))
    assert (pl.n_kept, pl.n_cached) == (2048, 2048)
    pl = oc.plan(oc.Shape(25, 72, 128, 320, 5, 64), oc.Cfg("frame_token", r=0.5, r_frame=0.2))
    assert (pl.n_frame_cached, pl.n_seq, pl.seq_len, pl.n_cached) == (5, 20, 4608, 138240)
    pl = oc.plan(oc.Shape(16, 16, 16, 1152, 16, 72), oc.Cfg("block", r=0.5))
    assert (pl.n_seq, pl.seq_len) == (128, 16)


def _status(fn):
    with pytest.raises(oc.OmniCacheError) as e:
        fn()
    return e.value.status


GOOD = oc.Shape(1, 8, 8, 32, 2, 16, 0, "bf16")


@pytest.mark.parametrize("shape,cfg,status", [
    (oc.Shape(1, 8, 8, 32, 2, 16, 0, "bf16"), oc.Cfg("token", r=1.0), L.OC_ERR_INVALID_ARG),
    (oc.Shape(1, 8, 8, 32, 2, 16, 0, "bf16"), oc.Cfg("token", r=float("nan")), L.OC_ERR_INVALID_ARG),
    (oc.Shape(1, 8, 8, 32, 2, 16, 0, "bf16"), oc.Cfg("token", r=-0.1), L.OC_ERR_INVALID_ARG),
    (oc.Shape(1, 8, 8, 32, 2, 16, 0, "bf16"), oc.Cfg("token", r=0.5, patch_k=3), L.OC_ERR_SHAPE),
    (oc.Shape(1, 6, 8, 32, 2, 16, 0, "bf16"), oc.Cfg("token", r=0.5, patch_k=2), L.OC_ERR_SHAPE),
    (oc.Shape(1, 7, 8, 32, 2, 16, 0, "bf16"), oc.Cfg("token", r=0.5), L.OC_ERR_SHAPE),
    (oc.Shape(1, 8, 8, 30, 2, 16, 0, "bf16"), oc.Cfg("token", r=0.5), L.OC_ERR_SHAPE),
    (oc.Shape(1, 8, 8, 32, 2, 12, 0, "bf16"), oc.Cfg("token", r=0.5), L.OC_ERR_SHAPE),
    (oc.Shape(1, 8, 8, 32, 2, 24, 0, "bf16"), oc.Cfg("token", r=0.5), L.OC_ERR_SHAPE),
    (oc.Shape(1, 8, 8, 32, 2, 136, 0, "f32"), oc.Cfg("token", r=0.5), L.OC_ERR_SHAPE),
    (oc.Shape(2, 8, 8, 32, 2, 16, 3, "bf16"), oc.Cfg("token", r=0.5), L.OC_ERR_SHAPE),
    (oc.Shape(1, 8, 8, 32, 2, 16, 3, "bf16"), oc.Cfg("block", r=0.5), L.OC_ERR_SHAPE),
    (oc.Shape(1, 8, 8, 32, 2, 16, 0, "bf16"), oc.Cfg("frame", r_frame=0.5), L.OC_ERR_SHAPE),
    (oc.Shape(33, 8, 8, 32, 2, 16, 0, "bf16"), oc.Cfg("frame_token", r=0.5, r_frame=0.2), L.OC_ERR_SHAPE),
    (oc.Shape(4, 34, 34, 32, 2, 16, 0, "bf16"), oc.Cfg("frame", r_frame=0.2, patch_k=17), L.OC_ERR_SHAPE),
    (oc.Shape(1, 256, 256, 32, 2, 16, 0, "bf16"), oc.Cfg("token", r=0.5), L.OC_ERR_SHAPE),
])
def test_plan_rejects(shape, cfg, status):
    assert _status(lambda: oc.plan(shape, cfg)) == status
    assert L.lib().oc_last_error().decode() != ""


def test_plan_rejects_bad_enums_and_dtype():
    lib = L.lib()
    info = L.oc_plan_info()
    sh = GOOD.c()
    cf = oc.Cfg("token", r=0.5).c()
    cf.gran = 9
    assert lib.oc_plan(C.byref(sh), C.byref(cf), C.byref(info)) == L.OC_ERR_INVALID_ARG
    # a coarser level: Token and Block Cache only, coarse_k dividing patch_k
    # and smaller, its ratio in [0, 1)
    for bad, status in ((oc.Cfg("frame", r_frame=0.3, patch_k=2, coarse_k=1, r_coarse=0.1), L.OC_ERR_INVALID_ARG),
                        (oc.Cfg("token", r=0.3, patch_k=4, coarse_k=3, r_coarse=0.1), L.OC_ERR_SHAPE),
                        (oc.Cfg("token", r=0.3, patch_k=2, coarse_k=2, r_coarse=0.1), L.OC_ERR_SHAPE),
                        (oc.Cfg("token", r=0.3, patch_k=2, coarse_k=-1, r_coarse=0.1), L.OC_ERR_SHAPE),
                        (oc.Cfg("block", r=0.3, patch_k=2, coarse_k=1, r_coarse=1.0), L.OC_ERR_INVALID_ARG),
                        (oc.Cfg("block", r=0.3, patch_k=2, coarse_k=1, r_coarse=float("nan")), L.OC_ERR_INVALID_ARG)):
        cf = bad.c()
        assert lib.oc_plan(C.byref(sh), C.byref(cf), C.byref(info)) == status, bad
    cf = oc.Cfg("token", r=0.5).c()
    sh.dtype = 7
    assert lib.oc_plan(C.byref(sh), C.byref(cf), C.byref(info)) == L.OC_ERR_DTYPE
    assert lib.oc_plan(None, C.byref(cf), C.byref(info)) == L.OC_ERR_INVALID_ARG
    assert lib.oc_plan(C.byref(GOOD.c()), C.byref(cf), None) == L.OC_ERR_INVALID_ARG
    assert lib.oc_status_string(L.OC_ERR_WORKSPACE) == b"OC_ERR_WORKSPACE"


FAKE = 1 << 20   # an aligned, never dereferenced address: calls below fail validation first


def test_entry_points_validate_before_launching():
    lib = L.lib()
    sh = GOOD.c()
    cf = oc.Cfg("token", r=0.5).c()
    need = oc.plan(GOOD, oc.Cfg("token", r=0.5)).workspace_bytes
    # NULL input
    assert lib.oc_match(C.byref(sh), C.byref(cf), None, FAKE, FAKE, None, FAKE, need, None) == L.OC_ERR_INVALID_ARG
    # misaligned input
    assert lib.oc_match(C.byref(sh), C.byref(cf), FAKE + 2, FAKE, FAKE, None, FAKE, need, None) == L.OC_ERR_INVALID_ARG
    # workspace too small
    assert lib.oc_match(C.byref(sh), C.byref(cf), FAKE, FAKE, FAKE, None, FAKE, need - 1, None) == L.OC_ERR_WORKSPACE
    assert lib.oc_select(C.byref(sh), C.byref(cf), FAKE, FAKE, FAKE, FAKE, FAKE, 0, FAKE, 16, None) == L.OC_ERR_WORKSPACE
    assert lib.oc_select(C.byref(sh), C.byref(cf), FAKE, FAKE, FAKE, FAKE, FAKE, 2, FAKE, need, None) == \
        L.OC_ERR_INVALID_ARG
    assert lib.oc_gather(C.byref(sh), C.byref(cf), FAKE, FAKE, FAKE, None) == L.OC_ERR_INVALID_ARG   # aliasing
    w = L.oc_attn_weights(FAKE, FAKE, FAKE, None)
    assert lib.oc_attn_reduced(C.byref(sh), FAKE, 1, 4, None, C.byref(w), FAKE, None, FAKE, 1 << 30, None) == \
        L.OC_ERR_INVALID_ARG
    w = L.oc_attn_weights(FAKE, FAKE, FAKE, FAKE)
    assert lib.oc_attn_reduced(C.byref(sh), FAKE, 1, 4, None, C.byref(w), FAKE, None, FAKE, 16, None) == \
        L.OC_ERR_WORKSPACE
    ctx_shape = oc.Shape(1, 8, 8, 32, 2, 16, 3, "bf16").c()
    assert lib.oc_attn_reduced(C.byref(ctx_shape), FAKE, 2, 4, FAKE, C.byref(w), FAKE, FAKE, FAKE, 1 << 30, None) == \
        L.OC_ERR_SHAPE
    assert lib.oc_restore(C.byref(sh), FAKE, 4, None, None, FAKE, None) == L.OC_ERR_INVALID_ARG
    # cache state
    cache = L.oc_cache(None, 0, 0)
    assert lib.oc_layer_cached(C.byref(sh), C.byref(cf), FAKE, None, C.byref(w), C.byref(cache), None, None, FAKE,
                               need, None) == L.OC_ERR_CACHE_STATE
    cache = L.oc_cache(FAKE * 2, 3, 0)
    assert lib.oc_layer_cached(C.byref(sh), C.byref(cf), FAKE, None, C.byref(w), C.byref(cache), None, None, FAKE,
                               need, None) == L.OC_ERR_CACHE_STATE
    cache = L.oc_cache(FAKE, 1, 0)   # x aliases the cache
    assert lib.oc_layer_cached(C.byref(sh), C.byref(cf), FAKE, None, C.byref(w), C.byref(cache), None, None, FAKE,
                               need, None) == L.OC_ERR_INVALID_ARG
    assert cache.step == 0 and cache.valid == 1
    assert lib.oc_attn_full(C.byref(sh), C.byref(cf), FAKE, None, C.byref(w), FAKE * 2, None, FAKE, need - 1, None) == \
        L.OC_ERR_WORKSPACE


def test_workspace_covers_cold_full_steps():
    # the cold "full" step computes everything, so the workspace covers it
    for name, shape, cfg in WORKLOAD_SHAPES:
        need = oc.plan(shape, cfg).workspace_bytes
        full = oc.plan(shape, oc.Cfg(cfg.gran, 0.0, 0.0, cfg.patch_k)).workspace_bytes
        assert need >= full, name


def test_plan_and_errors_from_many_threads():
    """Host entry points called concurrently from several threads: every
    thread gets the same plan for the same arguments, and each thread's
    oc_last_error() holds the message of its own last failure (the error
    text is thread-local; the library's shared host state is guarded)."""
    import threading
    lib = L.lib()
    good_cf = oc.Cfg("token", r=0.5)
    ref = oc.plan(GOOD, good_cf)
    bad = oc.Shape(1, 8, 8, 30, 2, 16, 0, "bf16")           # C not a multiple of 8
    errors, results = [], []

    def worker(i):
        try:
            for it in range(200):
                if (i + it) % 2:
                    info = oc.plan(GOOD, good_cf)
                    results.append(info == ref)
                else:
                    sh, cf, info = bad.c(), good_cf.c(), L.oc_plan_info()
                    st = lib.oc_plan(C.byref(sh), C.byref(cf), C.byref(info))
                    msg = lib.oc_last_error().decode()
                    results.append(st == L.OC_ERR_SHAPE and "C=30" in msg)
        except Exception as e:   # pragma: no cover - reported below
            errors.append(repr(e))

    th = [threading.Thread(target=worker, args=(i,)) for i in range(8)]
    for t in th:
        t.start()
    for t in th:
        t.join()
    assert not errors, errors
    assert len(results) == 8 * 200 and all(results)


def test_static_entry_point_rejects_layers_beyond_its_scratch():
    """oc_layer_cached_static refuses, before any device work, a layer whose
    workspace exceeds the library's static scratch (the SVD-XT-sized level
    needs 576 MiB against 96 MiB), with a message naming both sizes."""
    lib = L.lib()
    big = oc.Shape(25, 72, 128, 320, 5, 64, 0, "bf16")
    cfg = oc.Cfg("frame_token", r=0.5, r_frame=0.2)
    need = oc.plan(big, cfg).workspace_bytes
    assert need > oc.static_scratch_bytes() == 96 << 20
    sh, cf = big.c(), cfg.c()
    w = L.oc_attn_weights(FAKE, FAKE, FAKE, FAKE)
    cache = L.oc_cache(FAKE * 2, 0, 0)
    st = lib.oc_layer_cached_static(C.byref(sh), C.byref(cf), FAKE, None, C.byref(w), C.byref(cache), None, None,
                                    None)
    assert st == L.OC_ERR_WORKSPACE
    msg = lib.oc_last_error().decode()
    assert str(need) in msg and str(96 << 20) in msg
    assert cache.valid == 0 and cache.step == 0


def test_ffn_entry_point_validates_before_launching():
    lib = L.lib()
    sh = oc.Shape(1, 8, 8, 64, 2, 32, 0, "bf16").c()
    need = lib.oc_ffn_workspace_bytes(C.byref(sh), 256, 32)
    assert need == 32 * 256 * 2 + 64 * 256 * 2
    w = L.oc_ffn_weights(FAKE, FAKE, 256, 0)
    ok_args = (C.byref(sh), FAKE, FAKE, 32, C.byref(w), FAKE * 2, 1, FAKE, need, None)
    assert lib.oc_ffn_reduced(*ok_args[:8], need - 1, None) == L.OC_ERR_WORKSPACE
    bad = L.oc_ffn_weights(FAKE, FAKE, 96, 0)                       # hidden not a multiple of 64
    assert lib.oc_ffn_reduced(C.byref(sh), FAKE, FAKE, 32, C.byref(bad), FAKE * 2, 1, FAKE, need, None) == \
        L.OC_ERR_SHAPE
    res = L.oc_ffn_weights(FAKE, FAKE, 256, 1)
    assert lib.oc_ffn_reduced(C.byref(sh), FAKE, FAKE, 32, C.byref(res), FAKE * 2, 1, FAKE, need, None) == \
        L.OC_ERR_INVALID_ARG
    assert lib.oc_ffn_reduced(C.byref(sh), FAKE, FAKE, 65, C.byref(w), FAKE * 2, 1, FAKE, 1 << 30, None) == \
        L.OC_ERR_SHAPE                                                # more rows than tokens
    assert lib.oc_ffn_reduced(C.byref(sh), FAKE, FAKE, 32, C.byref(w), FAKE, 1, FAKE, need, None) == \
        L.OC_ERR_INVALID_ARG                                          # y aliases x
    assert lib.oc_ffn_reduced(C.byref(sh), FAKE, FAKE, 32, C.byref(w), FAKE * 2, 2, FAKE, need, None) == \
        L.OC_ERR_INVALID_ARG
    f32 = oc.Shape(1, 8, 8, 64, 2, 32, 0, "f32").c()
    assert lib.oc_ffn_reduced(C.byref(f32), FAKE, FAKE, 32, C.byref(w), FAKE * 2, 1, FAKE, need, None) == \
        L.OC_ERR_DTYPE
    c72 = oc.Shape(1, 8, 8, 72, 2, 32, 0, "bf16").c()
    assert lib.oc_ffn_reduced(C.byref(c72), FAKE, FAKE, 32, C.byref(w), FAKE * 2, 1, FAKE, need, None) == \
        L.OC_ERR_SHAPE
    assert lib.oc_ffn_reduced(C.byref(sh), FAKE, FAKE, 0, C.byref(w), FAKE * 2, 1, FAKE, 0, None) == L.OC_OK


@pytest.mark.parametrize("gran,F,H,W,k1,k2,r1,r2", [
    ("token", 1, 64, 64, 4, 1, 0.25, 0.25), ("token", 2, 16, 16, 4, 2, 0.2, 0.3), ("token", 1, 32, 32, 8, 2, 0.3, 0.4),
    ("token", 1, 16, 16, 2, 1, 0.7, 0.7), ("block", 4, 16, 16, 4, 1, 0.25, 0.25), ("block", 6, 8, 16, 2, 1, 0.1, 0.5),
])
def test_plan_of_two_levels_matches_the_oracle(gran, F, H, W, k1, k2, r1, r2):
    """Host only: the plan of a two-level hierarchy (coarse_k) gives the
    sequence count, lengths and retained total of the oracle's decisions
    for the same configuration."""
    from oracle import oc_oracle as O
    sh = oc.Shape(F, H, W, 8, 1, 16, 0, "bf16")
    pl = oc.plan(sh, oc.Cfg(gran, r=r1, patch_k=k1, coarse_k=k2, r_coarse=r2))
    osh = O.LayerShape(F, H, W, 8, 1, 16)
    x = np.random.default_rng(1).standard_normal((F, H * W, 8))
    dec = O.decide(x, osh, O.CacheCfg(gran, r=r1, patch_k=k1, coarse_k=k2, r_coarse=r2))
    seqs = O.build_sequences(osh, O.CacheCfg(gran, r=r1, patch_k=k1, coarse_k=k2, r_coarse=r2), dec)
    assert pl.n_seq == len(seqs) and all(len(s) == pl.seq_len for s in seqs)
    assert pl.n_kept == sum(len(s) for s in seqs) and pl.n_cached == F * H * W - pl.n_kept
