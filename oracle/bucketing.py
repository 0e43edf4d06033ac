"""Optimal sequence bucketing by dynamic programming (paper Sec. III.A).

Test infrastructure only (see oracle/__init__.py).

The paper's objective: split the sequences, sorted by length, into Q buckets
(contiguous length ranges); every sequence of a bucket is padded to the
bucket's upper length, so the padded work is sum_b upper_b * count_b
(eq. 2 with the per-bucket cost of eq. 1; the DP's score).  The DP runs over
the length histogram f, where f[l] counts the sequences of length l.

How the printed text is read here (it is garbled in places):
  * The histogram is indexed by the length itself, with an empty entry for
    length 0, so the table's column i stands for "all sequences of length at
    most i" and the optimum sits in column Lmax; the procedure's bound on i
    and its starting point for the walk back are consistent only with this.
  * cost[q][i] = min over 0 <= j < i of cost[q-1][j] + i * (F[i] - F[j]), with
    F the inclusive prefix sum of f: the top range (j, i] of a q-range cover
    holds F[i] - F[j] sequences, each padded to i.  Only cost[0][0] = 0 is
    finite in row 0; unreachable predecessors are skipped.  (The notation
    list transposes the table's indices and garbles the summation bounds;
    the procedure's arithmetic is what is followed.)
  * Ties: the procedure scans split points downwards and only a strictly
    smaller score replaces the incumbent, so among equal minima the largest
    split point is kept.
  * Q larger than the number of distinct lengths D is clamped to D (every
    extra bucket would be empty); the clamped count is returned.
"""
from __future__ import annotations

import numpy as np

INF = np.iinfo(np.int64).max // 4


def length_histogram(lengths) -> np.ndarray:
    """f[l] = number of sequences of length l, for l = 0..Lmax (f[0] = 0)."""
    lengths = np.asarray(lengths, dtype=np.int64)
    if lengths.size == 0 or lengths.min() < 1:
        raise ValueError("lengths must be >= 1 and non-empty")
    return np.bincount(lengths, minlength=int(lengths.max()) + 1).astype(np.int64)


def dynamic_bucketing(Q: int, f: np.ndarray):
    """The recurrence above over every length 0..Lmax.  Row q of the table
    is filled from row q-1: for each end point i all split points j < i are
    scored at once, and the largest j reaching the minimum is recorded.
    Returns (bests, optimum): bests[b] is the upper length of bucket b, read
    back from column Lmax through the recorded split points."""
    Lmax = len(f) - 1
    F = np.cumsum(f).astype(np.int64)           # F[x] = sum_{t<=x} f[t]
    cost = np.full((Q + 1, Lmax + 1), INF, np.int64)
    split = np.full((Q + 1, Lmax + 1), -1, np.int64)
    cost[0, 0] = 0
    for q in range(1, Q + 1):
        below = cost[q - 1]
        for i in range(1, Lmax + 1):
            reach = below[:i] != INF            # split points j = 0..i-1
            if not reach.any():
                continue
            score = np.where(reach, np.where(reach, below[:i], 0) + i * (F[i] - F[:i]), INF)
            best = score.min()
            cost[q, i] = best
            split[q, i] = np.flatnonzero(score == best)[-1]
    bests = [Lmax]
    for q in range(Q, 1, -1):
        bests.append(int(split[q, bests[-1]]))
    return bests[::-1], int(cost[Q, Lmax])


def bucket_plan(lengths, K: int):
    """Lengths -> (bests, bucket_of, K_eff, padded_steps).

    bests[b] is the upper length of bucket b (strictly increasing, last =
    Lmax); bucket_of[s] is the smallest b with lengths[s] <= bests[b];
    padded_steps = sum_b bests[b] * count_b, the DP's optimum."""
    if K < 1:
        raise ValueError("K must be >= 1")
    lengths = np.asarray(lengths, dtype=np.int64)
    f = length_histogram(lengths)
    K_eff = min(K, int(np.count_nonzero(f)))
    bests, value = dynamic_bucketing(K_eff, f)
    bests = np.asarray(bests, np.int64)
    bucket_of = np.searchsorted(bests, lengths, side="left").astype(np.int32)
    counts = np.bincount(bucket_of, minlength=K_eff)
    padded = int(np.sum(bests * counts))
    assert padded == value
    return bests.astype(np.int32), bucket_of, K_eff, padded
