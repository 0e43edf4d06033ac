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
"""
from __future__ import annotations

import numpy as np


def epoch_batches(lengths, bucket_of, K_eff: int, keys, B: int):
    """Returns a list of int64 arrays, one per mini-batch, in training order;
    each holds sequence indices sorted by (length desc, index asc)."""
    lengths = np.asarray(lengths, np.int64)
    bucket_of = np.asarray(bucket_of, np.int64)
    keys = np.asarray(keys, np.uint64)
    batches = []
    for b in range(K_eff):
        members = [s for s in range(len(lengths)) if bucket_of[s] == b]
        members.sort(key=lambda s: (int(keys[s]), s))
        for start in range(0, len(members), B):
            chunk = members[start:start + B]
            chunk.sort(key=lambda s: (-int(lengths[s]), s))
            batches.append(np.asarray(chunk, np.int64))
    return batches


def padded_batch_steps(lengths, batches) -> int:
    """Sum over batches of batch size times its longest sequence (eq. 1 per
    batch): the timesteps a dense padded implementation computes."""
    lengths = np.asarray(lengths, np.int64)
    return int(sum(len(bt) * int(lengths[bt].max()) for bt in batches))
