"""Brute-force checks for tiny vocabularies, written independently of the oracle.

Used only by the oracle pin tests: each function spells out a definition in the most literal way
(enumeration over subsets, exact interval measure of the inverse CDF) so that the oracle's sort-based
implementation can be checked against it on inputs small enough to enumerate.
"""
from __future__ import annotations

import itertools
import math


def nucleus_by_enumeration(mass, p):
    """Smallest-cardinality subset of ``range(len(mass))`` whose normalised mass is >= p; among the
    subsets of that size the one with the largest mass (the nucleus of Holtzman et al., ICLR 2020).
    Requires distinct masses so the answer is unique."""
    n = len(mass)
    tot = math.fsum(mass)
    for size in range(1, n + 1):
        best = None
        for sub in itertools.combinations(range(n), size):
            s = math.fsum(mass[i] for i in sub) / tot
            if s >= p and (best is None or s > best[0]):
                best = (s, set(sub))
        if best is not None:
            return best[1]
    return set(range(n))


def topk_by_definition(z, k):
    """Ids whose value is at least the k-th largest value, counting duplicates."""
    if k <= 0 or k >= len(z):
        return set(i for i, v in enumerate(z) if v != -math.inf)
    kth = sorted(z, reverse=True)[k - 1]
    return set(i for i, v in enumerate(z) if v >= kth and v != -math.inf)


def minp_by_definition(z, min_p):
    """Ids whose probability is at least min_p times the largest probability (real arithmetic)."""
    m = max(z)
    return set(i for i, v in enumerate(z) if math.exp(v - m) >= min_p)


def draw_measure(draw, n_ids, grid=20000):
    """Fraction of u in a uniform grid over [0, 1) that ``draw(u)`` maps to each id."""
    counts = [0] * n_ids
    for j in range(grid):
        counts[draw((j + 0.5) / grid)] += 1
    return [c / grid for c in counts]
