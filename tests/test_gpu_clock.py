"""The shader clock sampler (oc_clock_sample), a measurement aid of the
benchmark: counters that advance, a clock within the chip's range, and the
argument checks of the C ABI."""
import pytest
import torch

import paper_2607_23844_amd as oc
from paper_2607_23844_amd import _lib as L

pytestmark = pytest.mark.gpu


def test_clock_sampler_reads_a_plausible_clock():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    dev = torch.device("cuda:0")
    n = 200
    buf = torch.zeros(2 * n, dtype=torch.int64, device=dev)
    oc.clock_sample(buf, n, 100)          # one reading per µs
    torch.cuda.synchronize()
    a = buf.view(-1, 2).cpu()
    assert bool((a[1:, 0] > a[:-1, 0]).all()) and bool((a[1:, 1] >= a[:-1, 1] + 100).all())
    ghz = oc.clock_ghz(buf)
    print(f"idle clock: median {float(sorted(ghz)[len(ghz) // 2]):.2f} GHz", flush=True)
    assert 0.3 < float(sorted(ghz)[len(ghz) // 2]) < 3.5


def test_clock_sampler_rejects_bad_arguments():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lib = L.lib()
    buf = torch.zeros(8, dtype=torch.int64, device=torch.device("cuda:0"))
    s = torch.cuda.current_stream().cuda_stream
    assert lib.oc_clock_sample(None, 4, 10, s) == L.OC_ERR_INVALID_ARG
    assert lib.oc_clock_sample(buf.data_ptr(), 0, 10, s) == L.OC_ERR_INVALID_ARG
    assert lib.oc_clock_sample(buf.data_ptr(), 4, -1, s) == L.OC_ERR_INVALID_ARG
    with pytest.raises(ValueError):
        oc.clock_sample(buf, 5, 10)
