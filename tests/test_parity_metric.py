"""The output error measure of the parity tests (rel_err) on constructed
cases: a correctly rounded bf16 result scores zero, an error beyond the
rounding is reported at its size relative to the RMS."""
import numpy as np

from oc_synth import bf16_bits
from parity import rel_err


def _round_bf16(a):
    return (bf16_bits(a.astype(np.float32)).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def test_correctly_rounded_bf16_scores_zero():
    rng = np.random.default_rng(0)
    ref = rng.standard_normal(4096) * np.exp(rng.uniform(-4, 4, 4096))
    assert rel_err(_round_bf16(ref), ref, "bf16") == 0.0
    # the same values read as fp32 outputs carry the whole rounding error
    assert rel_err(_round_bf16(ref), ref, "f32") > 1e-3


def test_error_beyond_rounding_is_measured():
    rng = np.random.default_rng(1)
    ref = rng.standard_normal(4096)
    rms = np.sqrt(np.mean(ref * ref))
    y = _round_bf16(ref)
    y[17] += 0.05 * rms
    e = rel_err(y, ref, "bf16")
    # the planted 5% error, moved by the element's own rounding (at most half
    # an ulp) and less the half ulp taken off
    h = 2.0 ** -9 * 2.0 ** np.ceil(np.log2(abs(ref[17]))) / rms
    assert 0.05 - 2 * h - 1e-12 <= e <= 0.05 + 1e-12
