"""Pins of the oracle's feed-forward sublayer (the SD3 experiments cache the
FFN under the same selection as attention, OmniCache §4.2 "Design
choices"): library routines in fp64, exact identities of the tanh GELU,
closed forms, and the restoration invariants shared with the attention
sublayer."""
import math

import numpy as np
import pytest
import torch

from oracle import oc_oracle as O
from oc_synth import small_workload


def test_gelu_matches_torch_tanh_gelu_fp64():
    u = np.linspace(-12.0, 12.0, 4001)
    ref = torch.nn.functional.gelu(torch.from_numpy(u), approximate="tanh").numpy()
    np.testing.assert_allclose(O.gelu_tanh(u), ref, rtol=2e-16, atol=1e-15)


def test_gelu_identities():
    """0.5u(1 + tanh a) - 0.5(-u)(1 + tanh(-a)) = u for every u (tanh is
    odd); GELU(0) = 0; GELU(u) -> u and GELU(-u) -> 0 for large u; and the
    tanh form stays within 5e-4 of the exact erf GELU (a wrong constant of
    the approximation breaks this: its largest deviation is 4.73e-4)."""
    u = np.linspace(-8.0, 8.0, 1601)
    np.testing.assert_allclose(O.gelu_tanh(u) - O.gelu_tanh(-u), u, rtol=0, atol=1e-14)
    assert O.gelu_tanh(np.array([0.0]))[0] == 0.0
    assert abs(O.gelu_tanh(np.array([30.0]))[0] - 30.0) < 1e-12
    assert abs(O.gelu_tanh(np.array([-30.0]))[0]) < 1e-12
    erf = np.array([0.5 * v * (1.0 + math.erf(v / math.sqrt(2.0))) for v in u])
    assert np.max(np.abs(O.gelu_tanh(u) - erf)) < 5e-4


def test_feed_forward_matches_torch_linear_fp64():
    rng = np.random.default_rng(3)
    X = rng.standard_normal((37, 24))
    w1 = rng.standard_normal((96, 24)) / math.sqrt(24)
    w2 = rng.standard_normal((24, 96)) / math.sqrt(96)
    t = torch.from_numpy
    ref = torch.nn.functional.linear(torch.nn.functional.gelu(torch.nn.functional.linear(t(X), t(w1)),
                                                              approximate="tanh"), t(w2)).numpy()
    np.testing.assert_allclose(O.feed_forward(X, w1, w2), ref, rtol=0, atol=1e-13)


def test_feed_forward_diagonal_closed_form():
    """W1 = diag(a), W2 = I: each output channel is GELU(a_c x_c) of its own
    input channel alone."""
    rng = np.random.default_rng(4)
    C = 16
    a = rng.uniform(-3, 3, C)
    X = rng.standard_normal((5, C))
    y = O.feed_forward(X, np.diag(a), np.eye(C))
    for i in range(5):
        for c in range(C):
            v = a[c] * X[i, c]
            assert y[i, c] == pytest.approx(0.5 * v * (1 + math.tanh(math.sqrt(2 / math.pi) * (v + 0.044715 * v ** 3))),
                                            abs=1e-15)


@pytest.mark.parametrize("gran,F", [(O.TOKEN, 1), (O.BLOCK, 4), (O.FRAME, 6)])
def test_ffn_step_restoration(gran, F):
    """Under the attention's selection: with nothing cached the FFN step is
    the plain map of every row; on a warm step retained rows are fresh and
    cached rows carry the previous step's values; on a cold "matched" step a
    cached row equals the fresh row of the position its best match occupies."""
    wl = small_workload(gran, F=F, H=8, W=8, C=16, heads=2, head_dim=8, seed=23, r=0.5, r_frame=0.35,
                        planted=gran == O.FRAME)
    shape = O.LayerShape(wl.F, wl.H, wl.W, wl.C, wl.heads, wl.head_dim)
    x = wl.f64(wl.steps[0]).reshape(F, wl.N, wl.C)
    rng = np.random.default_rng(5)
    w1 = rng.standard_normal((64, 16)) / 4.0
    w2 = rng.standard_normal((16, 64)) / 8.0
    xf = x.reshape(-1, wl.C)
    full = O.feed_forward(xf, w1, w2)
    FN = F * wl.N
    np.testing.assert_array_equal(O.ffn_step(xf, np.arange(FN), np.arange(FN), w1, w2, None), full)
    cfg = O.CacheCfg(gran, r=0.5, r_frame=0.35)
    dec = O.decide(x, shape, cfg)
    seqs = O.build_sequences(shape, cfg, dec)
    kept, cached, wmap = O.kept_and_map(shape, cfg, dec, seqs, cache_valid=True)
    _, _, cmap = O.kept_and_map(shape, cfg, dec, seqs, cache_valid=False)
    assert len(cached) > 0
    prev = rng.standard_normal((FN, wl.C))
    yw = O.ffn_step(xf, kept, wmap, w1, w2, prev)
    np.testing.assert_array_equal(yw[kept], full[kept])
    np.testing.assert_array_equal(yw[cached], prev[cached])
    yc = O.ffn_step(xf, kept, cmap, w1, w2, None)
    np.testing.assert_array_equal(yc[kept], full[kept])
    for p in cached:
        np.testing.assert_array_equal(yc[p], full[kept[cmap[p]]])
