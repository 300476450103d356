"""Layered Cache schedule proposal (OmniCache §3.4, Alg. 1): the oracle.

TEST INFRASTRUCTURE ONLY: used by the tests and the benchmark's CPU leg,
never by the product path; shares no code with the library.

Given, for each candidate layer-timestep pair (l, t), the latency L[l,t]
that caching there saves and the quality loss Q[l,t] it costs, a target
speed-up s_r and a cache interval N, Alg. 1 scores each pair by
w = Q / L (quality lost per unit of saved latency), walks the candidates
from the lowest score up, and keeps adding them, each as (l, t, N), until
the saved latency reaches the budget (1 - 1/s_r) * sum of L over the
candidates.

Readings where the algorithm leaves details open:
  L1  Candidates are listed layer-major (l, then t); equal scores keep that
      order (a stable sort), and every sum runs in that order.
  L2  The budget sums L over the candidate set P itself (as printed), so a
      masked-out pair contributes nothing to it.
  L3  The walk stops as soon as the saved latency is at least the budget,
      or when no candidate is left.
  L4  s_r >= 1 (a speed-up below 1 asks for no saving), every candidate has
      L > 0 and a finite Q, and N >= 1; N is attached to each chosen pair
      unchanged.
"""
from __future__ import annotations

import math
from typing import List, Optional, Sequence, Tuple

import numpy as np


def candidates(n_layers: int, n_steps: int, mask: Optional[np.ndarray] = None) -> List[Tuple[int, int]]:
    """The candidate pairs P in layer-major order (L1), optionally masked."""
    out = []
    for l in range(n_layers):
        for t in range(n_steps):
            if mask is None or mask[l, t]:
                out.append((l, t))
    return out


def schedule(lat: np.ndarray, qual: np.ndarray, target_speedup: float, interval: int,
             mask: Optional[np.ndarray] = None) -> Tuple[List[Tuple[int, int, int]], float, float]:
    """Alg. 1: returns (chosen (l, t, N) in selection order, saved latency,
    budget)."""
    lat = np.asarray(lat, dtype=np.float64)
    qual = np.asarray(qual, dtype=np.float64)
    assert target_speedup >= 1.0 and interval >= 1
    P = candidates(lat.shape[0], lat.shape[1], mask)
    for l, t in P:
        assert lat[l, t] > 0.0 and math.isfinite(qual[l, t])
    # score per candidate, then the candidates from the lowest score up
    w = [qual[l, t] / lat[l, t] for l, t in P]
    order = sorted(range(len(P)), key=lambda i: w[i])          # stable: ties keep layer-major order
    total = 0.0
    for l, t in P:
        total += lat[l, t]
    budget = (1.0 - 1.0 / target_speedup) * total
    saved = 0.0
    chosen = []
    it = iter(order)
    while saved < budget:
        i = next(it, None)
        if i is None:
            break
        l, t = P[i]
        chosen.append((l, t, interval))
        saved += lat[l, t]
    return chosen, saved, budget
