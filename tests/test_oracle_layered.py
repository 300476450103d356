"""Pins of the Layered Cache schedule oracle (OmniCache §3.4, Alg. 1): a
hand-worked example, and properties that any correct greedy of Alg. 1 has
(tested on seeded random tables): the chosen pairs are a prefix of the
candidates by increasing score, the shortest one whose latency reaches the
budget; larger speed-ups extend the schedule; scaling L or Q by a power of
two leaves it unchanged; s_r = 1 chooses nothing and a huge s_r everything."""
import json
import os

import numpy as np
import pytest

from oracle import layered as Ly

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "layered_alg1_worked.json")


def test_golden_alg1():
    g = json.load(open(GOLDEN))
    L, Q = np.array(g["latency"], float), np.array(g["quality"], float)
    for c in g["cases"]:
        mask = None
        if "mask_out" in c:
            mask = np.ones(L.shape, bool)
            for l, t in c["mask_out"]:
                mask[l, t] = False
        chosen, saved, budget = Ly.schedule(L, Q, c["s_r"], g["interval"], mask)
        assert [(l, t) for l, t, _ in chosen] == [tuple(p) for p in c["chosen"]]
        assert all(n == g["interval"] for _, _, n in chosen)
        assert saved == c["saved"]
        if "budget" in c:
            assert budget == c["budget"]


def _table(seed, n_layers=6, n_steps=7):
    rng = np.random.default_rng(seed)
    L = rng.uniform(0.5, 3.0, (n_layers, n_steps))
    Q = rng.uniform(0.0, 2.0, (n_layers, n_steps))
    Q[rng.random((n_layers, n_steps)) < 0.2] = 0.0          # free pairs (score 0: ties)
    return L, Q


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("s_r", [1.1, 1.5, 2.0, 3.7])
def test_greedy_prefix_properties(seed, s_r):
    L, Q = _table(seed)
    chosen, saved, budget = Ly.schedule(L, Q, s_r, 2)
    P = Ly.candidates(*L.shape)
    w = {p: Q[p] / L[p] for p in P}
    pairs = [(l, t) for l, t, _ in chosen]
    # every chosen pair scores no higher than any unchosen one
    rest = [p for p in P if p not in set(pairs)]
    if pairs and rest:
        assert max(w[p] for p in pairs) <= min(w[p] for p in rest)
    # scores are non-decreasing along the selection, ties in layer-major order
    for a, b in zip(pairs, pairs[1:]):
        assert w[a] < w[b] or (w[a] == w[b] and a < b)
    # the shortest such prefix reaching the budget
    assert saved >= budget and saved - L[pairs[-1]] < budget
    assert budget == pytest.approx((1 - 1 / s_r) * L.sum(), rel=1e-15)


@pytest.mark.parametrize("seed", range(4))
def test_monotone_in_speedup_and_extremes(seed):
    L, Q = _table(seed)
    prev = []
    for s_r in (1.0, 1.05, 1.3, 2.0, 5.0, 1e12):
        chosen, _, _ = Ly.schedule(L, Q, s_r, 1)
        assert chosen[:len(prev)] == prev
        prev = chosen
    assert Ly.schedule(L, Q, 1.0, 1)[0] == []
    assert len(Ly.schedule(L, Q, 1e12, 1)[0]) == L.size


@pytest.mark.parametrize("seed", range(4))
def test_power_of_two_scaling_invariance(seed):
    L, Q = _table(seed)
    base = Ly.schedule(L, Q, 2.5, 4)[0]
    assert Ly.schedule(L * 8.0, Q, 2.5, 4)[0] == base
    assert Ly.schedule(L, Q * 0.25, 2.5, 4)[0] == base


# ----------------------------------------------------------------------------
# the library's implementation against the oracle (host code, no GPU)
# ----------------------------------------------------------------------------

def test_library_matches_oracle_on_golden_and_tables():
    import paper_2607_23844_amd as oc
    from oc_synth import layered_tables
    g = json.load(open(GOLDEN))
    L, Q = np.array(g["latency"], float), np.array(g["quality"], float)
    cases = [(L, Q, c["s_r"], g["interval"], None) for c in g["cases"] if "mask_out" not in c]
    mask = np.ones(L.shape, bool)
    mask[1, 1] = False
    cases.append((L, Q, 2.0, 3, mask))
    for seed in range(4):
        Ls, Qs = layered_tables(seed=3000 + seed)
        m = np.random.default_rng(seed).random(Ls.shape) < 0.8
        for s_r in (1.0, 1.2, 1.75, 2.5, 4.0):
            cases.append((Ls, Qs, s_r, 1 + seed, None))
            cases.append((Ls, Qs, s_r, 2, m))
    for Lt, Qt, s_r, N, mk in cases:
        ref = Ly.schedule(Lt, Qt, s_r, N, mk)
        got = oc.layered_schedule(Lt, Qt, s_r, N, mk)
        assert got[0] == ref[0]
        assert got[1] == ref[1] and got[2] == ref[2]          # same sums in the same order: bit-identical


def test_library_rejects_bad_tables():
    import paper_2607_23844_amd as oc
    from paper_2607_23844_amd import _lib as L
    Lt = np.ones((2, 3))
    Qt = np.ones((2, 3))
    for bad in (dict(target_speedup=0.5), dict(interval=0)):
        kw = dict(target_speedup=2.0, interval=1)
        kw.update(bad)
        with pytest.raises(L.OmniCacheError) as e:
            oc.layered_schedule(Lt, Qt, **kw)
        assert e.value.status == L.OC_ERR_INVALID_ARG
    L0 = Lt.copy()
    L0[1, 2] = 0.0
    with pytest.raises(L.OmniCacheError):
        oc.layered_schedule(L0, Qt, 2.0, 1)
    m = np.ones((2, 3), bool)
    m[1, 2] = False                                            # a masked pair may hold anything
    assert oc.layered_schedule(L0, Qt, 2.0, 1, m)[0]
    Qn = Qt.copy()
    Qn[0, 0] = np.nan
    with pytest.raises(L.OmniCacheError):
        oc.layered_schedule(Lt, Qn, 2.0, 1)
