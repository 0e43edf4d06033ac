"""Brute-force optimal bucketing: enumerate every split of the sorted distinct
lengths into K contiguous non-empty groups.  Used only to pin the oracle and
the library's planner; independent of both."""
import itertools

import numpy as np


def brute_force(lengths, K):
    """Returns (best_cost, chosen_bests) where chosen_bests is the optimal
    partition whose upper bounds, read from the top bucket down, are
    lexicographically largest (the DP's tie rule)."""
    lengths = np.asarray(lengths, np.int64)
    vals, counts = np.unique(lengths, return_counts=True)
    D = len(vals)
    K = min(K, D)
    best_cost, best_key, best_bests = None, None, None
    for cuts in itertools.combinations(range(1, D), K - 1):
        edges = (0,) + cuts + (D,)
        cost = 0
        bests = []
        for a, b in zip(edges[:-1], edges[1:]):
            upper = int(vals[b - 1])
            cost += upper * int(counts[a:b].sum())
            bests.append(upper)
        key = tuple(reversed(bests))
        if best_cost is None or cost < best_cost or (cost == best_cost and key > best_key):
            best_cost, best_key, best_bests = cost, key, bests
    return best_cost, best_bests
