"""The C ABI without the Python binding: tests/c_abi/layer_chain.c plans a
layer, allocates the workspace, and runs a chain of cached steps carrying
the layer cache (OmniCache §3.2), using nothing but include/oc.h and
liboc.so.  On the CPU it must compile warning-free against the header as C;
on the GPU its outputs must equal, bit for bit, the same chain run through
the Python binding."""
import os
import struct
import subprocess
import sys

import numpy as np
import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
from oc_synth import make_workload, small_workload  # noqa: E402
import paper_2607_23844_amd as oc  # noqa: E402
from parity import dev_tensor, shapes, weights_dev  # noqa: E402

SRC = os.path.join(ROOT, "tests", "c_abi", "layer_chain.c")
EXE = os.path.join(ROOT, "tests", "c_abi", "layer_chain")
GRANS = {"token": 0, "frame": 1, "block": 2, "frame_token": 3}


def test_c_program_compiles_against_the_header(tmp_path):
    """The header is plain C and the example uses only what it declares."""
    out = tmp_path / "layer_chain"
    r = subprocess.run(["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-Werror", "-pedantic-errors",
                        "-D__HIP_PLATFORM_AMD__", "-isystem", "/opt/rocm/include", "-I", os.path.join(ROOT, "include"), SRC,
                        "-c", "-o", str(out) + ".o"], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def _write_input(path, wl, sh, cf, n_steps):
    esz = 2 if wl.dtype == "bf16" else 4
    with open(path, "wb") as f:
        f.write(struct.pack("<14i", sh.F, sh.H, sh.W, sh.C, sh.heads, sh.head_dim, sh.n_ctx,
                            1 if wl.dtype == "bf16" else 0, GRANS[cf.gran], cf.patch_k,
                            0 if cf.cold == "matched" else 1, n_steps, esz, cf.coarse_k))
        f.write(struct.pack("<3d", cf.r, cf.r_frame, cf.r_coarse))
        for a in [wl.wq, wl.wk, wl.wv, wl.wo] + ([wl.ctx] if wl.n_ctx else []) + list(wl.steps[:n_steps]):
            f.write(np.ascontiguousarray(a).tobytes())
    return esz


def _case(wl, tmp_path, name, n_steps):
    if not os.path.exists(EXE):
        pytest.fail(f"{EXE} is not built: run __graft_entry__.build()")
    sh, cf, _, _ = shapes(wl)
    inp, outp = tmp_path / f"{name}.in", tmp_path / f"{name}.out"
    esz = _write_input(inp, wl, sh, cf, n_steps)
    print(f"C chain {name}", flush=True)
    r = subprocess.run([EXE, str(inp), str(outp)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    FN = sh.F * sh.H * sh.W
    per = (FN + sh.n_ctx) * sh.C * esz
    raw = np.fromfile(outp, dtype=np.uint8)
    assert raw.size == per * n_steps
    # the same chain through the binding
    dev = torch.device("cuda:0")
    W = weights_dev(wl)
    ctx = dev_tensor(wl, wl.ctx) if wl.n_ctx else None
    cache = oc.LayerCache(sh, dev)
    ws = oc.workspace(sh, cf, dev)
    ity = np.uint16 if esz == 2 else np.uint32
    for s in range(n_steps):
        y, y_ctx, _ = oc.layer_cached(dev_tensor(wl, wl.steps[s]), W, cache, sh, cf, ctx=ctx, ws=ws)
        torch.cuda.synchronize()
        got = raw[s * per:(s + 1) * per].view(ity)
        want = y.view(torch.int16 if esz == 2 else torch.int32).cpu().numpy().view(ity).reshape(-1)
        np.testing.assert_array_equal(got[:FN * sh.C], want, err_msg=f"{name} step {s}: y")
        if wl.n_ctx:
            wc = y_ctx.view(torch.int16 if esz == 2 else torch.int32).cpu().numpy().view(ity).reshape(-1)
            np.testing.assert_array_equal(got[FN * sh.C:], wc, err_msg=f"{name} step {s}: y_ctx")


@pytest.mark.gpu
@pytest.mark.parametrize("kw", [
    dict(gran="token", F=1, H=16, W=16, C=128, heads=2, head_dim=64, dtype="bf16", n_ctx=5),
    dict(gran="frame_token", F=7, H=8, W=8, C=64, heads=2, head_dim=32, dtype="bf16", r_frame=0.3),
    dict(gran="block", F=9, H=8, W=8, C=64, heads=2, head_dim=32, dtype="f32"),
], ids=["token_ctx_bf16", "frame_token_bf16", "block_f32"])
def test_c_chain_matches_binding_small(kw, tmp_path):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    kw = dict(kw)
    wl = small_workload(kw.pop("gran"), n_steps=3, seed=5, **kw)
    _case(wl, tmp_path, wl.gran, 3)


@pytest.mark.gpu
def test_c_chain_matches_binding_sd3(tmp_path):
    """The benchmarked layer (4096 image + 333 text tokens, C = 1536, Token
    Cache r = 0.5), three steps."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    _case(make_workload("sd3_1024", 3), tmp_path, "sd3_1024", 3)
