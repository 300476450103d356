"""Concurrent first calls from several host threads (the library's shared
host state is the mutex-guarded record of kernels whose dynamic-LDS limit it
raised on each device).  Run in a fresh child process so that the calls
really are the first ones of that process; each thread has its own stream,
workspace and layer cache, and every thread's output must equal, bit for
bit, the same layer computed serially afterwards."""
import os
import subprocess
import sys
import threading

import pytest
import torch

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _child() -> int:
    sys.path.insert(0, ROOT)
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    from oc_synth import make_workload, small_workload
    import paper_2607_23844_amd as oc
    from parity import dev_tensor, shapes, weights_dev

    dev = torch.device("cuda:0")
    # the SD3-like layer (its Q/K/V projection uses tiles above 64 KB of LDS)
    # and a head-dim-64 temporal layer (the fused short-sequence kernel)
    layers = [make_workload("sd3_1024", 1),
              small_workload("block", F=16, H=16, W=16, C=128, heads=2, head_dim=64, dtype="bf16", seed=5)]
    setups = []
    for wl in layers:
        sh, cf, _, _ = shapes(wl)
        ctx = dev_tensor(wl, wl.ctx) if wl.n_ctx else None
        setups.append((sh, cf, dev_tensor(wl, wl.steps[0]), weights_dev(wl), ctx))
    torch.cuda.synchronize()
    n_threads = 4
    outs = [[None] * len(setups) for _ in range(n_threads)]
    errs = []
    gate = threading.Barrier(n_threads)

    def worker(i):
        try:
            s = torch.cuda.Stream(device=dev)
            with torch.cuda.stream(s):
                work = [(oc.workspace(sh, cf, dev), oc.LayerCache(sh, dev)) for sh, cf, _, _, _ in setups]
                torch.cuda.synchronize()
                gate.wait()
                for j, ((sh, cf, x, W, ctx), (ws, cache)) in enumerate(zip(setups, work)):
                    y, _, _ = oc.layer_cached(x, W, cache, sh, cf, ctx=ctx, ws=ws)
                    outs[i][j] = y
                s.synchronize()
        except Exception as e:
            errs.append(f"thread {i}: {e!r}")

    th = [threading.Thread(target=worker, args=(i,)) for i in range(n_threads)]
    for t in th:
        t.start()
    for t in th:
        t.join()
    if errs:
        print("\n".join(errs), flush=True)
        return 1
    for j, (sh, cf, x, W, ctx) in enumerate(setups):
        cache = oc.LayerCache(sh, dev)
        y, _, _ = oc.layer_cached(x, W, cache, sh, cf, ctx=ctx)
        torch.cuda.synchronize()
        for i in range(n_threads):
            if not torch.equal(outs[i][j].view(torch.int16), y.view(torch.int16)):
                print(f"layer {j}: thread {i} differs from the serial call", flush=True)
                return 1
    print("concurrent first calls: all threads bit-identical to the serial calls", flush=True)
    return 0


def test_concurrent_first_calls_from_threads():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    r = subprocess.run([sys.executable, os.path.abspath(__file__), "child"], capture_output=True, text=True,
                       timeout=300, cwd=ROOT)
    print(r.stdout[-2000:], r.stderr[-2000:], flush=True)
    assert r.returncode == 0


if __name__ == "__main__" and len(sys.argv) > 1 and sys.argv[1] == "child":
    sys.exit(_child())
