"""Optimal sequence bucketing by dynamic programming (paper Sec. III.A).

Test infrastructure only (see oracle/__init__.py).

The paper's objective: split the sequences, sorted by length, into Q buckets
(contiguous length ranges); every sequence of a bucket is padded to the
bucket's upper length, so the padded work is sum_b upper_b * count_b
(eq. 2 with the per-bucket cost of eq. 1; the DP's score).  The DP runs over
the length histogram f, where f[l] counts the sequences of length l.

Readings of the garbled text, applied here:
  * f is indexed by length, f[0] = 0, and the DP's index i runs over lengths
    1..Lmax; the answer is dp[Q][Lmax] (the pseudo-code's "n <- length(f)"
    and "curId <- n-1" only agree with this indexing).
  * dp[q][i] = min over 0 <= j < i of dp[q-1][j] + i * sum_{t=j+1..i} f[t];
    dp[0][0] = 0, every other entry starts at INF, and INF predecessors are
    skipped (the notation list's dp[i][k] is the transposed name of the same
    table, and its summation bounds are garbled).
  * ties: j runs downwards and only a strictly smaller value replaces the
    incumbent, so the largest minimising j wins.
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


def dynamic_bucketing_loops(Q: int, f: np.ndarray):
    """The DYNAMICBUCKETING procedure written as plain loops, in the paper's
    order (q outer, i middle, j descending inner, running sum of f).
    Returns (bests, dp_value).  O(Q * Lmax^2) Python steps: small inputs only."""
    Lmax = len(f) - 1
    dp = [[INF] * (Lmax + 1) for _ in range(Q + 1)]
    prev = [[-1] * (Lmax + 1) for _ in range(Q + 1)]
    dp[0][0] = 0
    for q in range(1, Q + 1):
        for i in range(1, Lmax + 1):
            cur = int(f[i])
            for j in range(i - 1, -1, -1):
                if dp[q - 1][j] != INF:
                    val = cur * i + dp[q - 1][j]
                    if val < dp[q][i]:
                        dp[q][i] = val
                        prev[q][i] = j
                cur += int(f[j])
    bests = []
    cur_id = Lmax
    for q in range(Q, 0, -1):
        bests.insert(0, cur_id)
        cur_id = prev[q][cur_id]
    return bests, dp[Q][Lmax]


def dynamic_bucketing(Q: int, f: np.ndarray):
    """Same DP as ``dynamic_bucketing_loops``; the inner j loop is evaluated as
    one vector expression.  The running sum of the j loop equals
    F[i] - F[j] with F the inclusive prefix sum of f, and "largest j among the
    minima" is the first minimum when j is scanned downwards.
    Returns (bests, dp_value)."""
    Lmax = len(f) - 1
    F = np.cumsum(f).astype(np.int64)           # F[x] = sum_{t<=x} f[t]
    dp = np.full((Q + 1, Lmax + 1), INF, np.int64)
    prev = np.full((Q + 1, Lmax + 1), -1, np.int64)
    dp[0, 0] = 0
    for q in range(1, Q + 1):
        for i in range(1, Lmax + 1):
            js = np.arange(i - 1, -1, -1)        # j = i-1 down to 0
            base = dp[q - 1, js]
            ok = base != INF
            if not ok.any():
                continue
            val = np.where(ok, (F[i] - F[js]) * i + np.where(ok, base, 0), INF)
            k = int(np.argmin(val))              # first minimum = largest j
            if val[k] < dp[q, i]:
                dp[q, i] = val[k]
                prev[q, i] = js[k]
    bests = []
    cur_id = Lmax
    for q in range(Q, 0, -1):
        bests.insert(0, int(cur_id))
        cur_id = prev[q, cur_id]
    return bests, int(dp[Q, Lmax])


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
