"""Per-epoch mini-batch schedule over the buckets (paper Sec. III, IV.A).

Test infrastructure only (see oracle/__init__.py).

The paper feeds each epoch bucket by bucket, shortest bucket first, and the
data are reshuffled before every epoch; with one bucket this is the paper's
unbucketed baseline, a purely random split into mini-batches.  Readings:
  * inside a bucket the shuffle is "sort by a random key" (keys are inputs,
    one per sequence per epoch; equal keys fall back to the sequence index),
  * consecutive runs of B shuffled sequences form the batches; the last,
    partial batch of a bucket is kept,
  * each batch is ordered by length, longest first (equal lengths by
    sequence index), so the sequences still running at step t are a prefix.
The paper leaves other feeding orders to future work (Sec. V); the ones here
(descending, whole buckets in random order, all batches interleaved at
random) are this library's definitions, pinned by hand-worked cases and by
invariants: every ordering feeds the same batches.
"""
from __future__ import annotations

import numpy as np


ORDERINGS = ("ascending", "descending", "random_buckets", "shuffled_batches")


def epoch_batches(lengths, bucket_of, K_eff: int, keys, B: int,
                  ordering: str = "ascending", order_keys=None):
    """Returns a list of int64 arrays, one per mini-batch, in training order;
    each holds sequence indices sorted by (length desc, index asc).

    `ordering` picks the order in which the batches are fed (the paper feeds
    the shortest bucket first and names other orders as future work, Sec. IV.A
    and Sec. V):
      ascending         bucket 0, 1, ..., K_eff-1 (the paper's order),
      descending        bucket K_eff-1, ..., 0,
      random_buckets    buckets sorted by (order_keys[b], b): whole buckets in
                        a random order,
      shuffled_batches  the ascending list of batches sorted by
                        (order_keys[i], i), i the batch's ascending position:
                        batches from all buckets interleaved at random.
    The batches themselves are the same in every ordering."""
    if ordering not in ORDERINGS:
        raise ValueError(f"unknown ordering {ordering!r}")
    lengths = np.asarray(lengths, np.int64)
    bucket_of = np.asarray(bucket_of, np.int64)
    keys = np.asarray(keys, np.uint64)
    per_bucket = []
    for b in range(K_eff):
        members = [s for s in range(len(lengths)) if bucket_of[s] == b]
        members.sort(key=lambda s: (int(keys[s]), s))
        chunks = []
        for start in range(0, len(members), B):
            chunk = members[start:start + B]
            chunk.sort(key=lambda s: (-int(lengths[s]), s))
            chunks.append(np.asarray(chunk, np.int64))
        per_bucket.append(chunks)
    if ordering == "descending":
        per_bucket = per_bucket[::-1]
    elif ordering == "random_buckets":
        ok = np.asarray(order_keys, np.uint64)
        rank = sorted(range(K_eff), key=lambda b: (int(ok[b]), b))
        per_bucket = [per_bucket[b] for b in rank]
    batches = [c for chunks in per_bucket for c in chunks]
    if ordering == "shuffled_batches":
        ok = np.asarray(order_keys, np.uint64)
        rank = sorted(range(len(batches)), key=lambda i: (int(ok[i]), i))
        batches = [batches[i] for i in rank]
    return batches


def padded_batch_steps(lengths, batches) -> int:
    """Sum over batches of batch size times its longest sequence (eq. 1 per
    batch): the timesteps a dense padded implementation computes."""
    lengths = np.asarray(lengths, np.int64)
    return int(sum(len(bt) * int(lengths[bt].max()) for bt in batches))
