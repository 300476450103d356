"""Brute-force checkers for tiny inputs.  TEST INFRASTRUCTURE ONLY.

These re-derive matching and selection with pure-Python loops and exact
rational arithmetic, independently of the NumPy oracle, so that tests can pin
the oracle to the definitions of OmniCache §3.2 (cosine matching, the r most
redundant candidates) rather than to itself.
"""
from __future__ import annotations

import itertools
import math
from fractions import Fraction
from typing import Dict, List, Sequence, Tuple


def dot(u: Sequence[float], v: Sequence[float]) -> float:
    return math.fsum(a * b for a, b in zip(u, v))


def cos_exact_order(u: Sequence[float], v: Sequence[float]) -> float:
    """Cosine with exactly rounded dot products (math.fsum); 0 for a
    zero-norm vector."""
    nu = math.sqrt(dot(u, u))
    nv = math.sqrt(dot(v, v))
    if nu == 0.0 or nv == 0.0:
        return 0.0
    return dot(u, v) / (nu * nv)


def brute_best_match(desc: Dict[int, Sequence[float]], src: Sequence[int],
                     dst: Sequence[int]) -> Tuple[Dict[int, float], Dict[int, int]]:
    """For every candidate, scan every representative; keep the first
    (smallest id) of the largest similarity."""
    best_v, best_i = {}, {}
    for s in src:
        bv, bi = None, None
        for d in sorted(dst):
            c = cos_exact_order(desc[s], desc[d])
            if bv is None or c > bv:
                bv, bi = c, d
        best_v[s], best_i[s] = bv, bi
    return best_v, best_i


def brute_select(node_max: Dict[int, float], R: int) -> List[int]:
    """Among all R-subsets of candidates, the one with the largest exact sum
    of best-match similarities; ties go to the lexicographically smallest
    sorted id tuple."""
    ids = sorted(node_max)
    best_sum, best_set = None, None
    for comb in itertools.combinations(ids, R):
        s = sum((Fraction(node_max[i]) for i in comb), Fraction(0))
        if best_sum is None or s > best_sum or (s == best_sum and comb < best_set):
            best_sum, best_set = s, comb
    return list(best_set) if best_set is not None else []


def brute_pairs(order: Sequence[int], sim: Dict[Tuple[int, int], float],
                dst: Sequence[int]) -> List[Tuple[int, int]]:
    """Greedy one-to-one pairing written as a repeated arg-max over a masked
    table (an independent formulation of the pairing rule)."""
    free = sorted(dst)
    out = []
    for s in order:
        vals = [(sim[(s, d)], -d) for d in free]
        v, negd = max(vals)
        d = -negd
        free.remove(d)
        out.append((s, d))
    return out
