"""Pins of the bucketing oracle (paper Sec. III.A, DYNAMICBUCKETING).

The DP reaches the exact optimum of its score, so it is pinned against the
plain definition (brute force over every contiguous partition), a hand-worked
example, and invariants that any correct implementation satisfies."""
import json
import os

import numpy as np
import pytest

from oracle import bucketing as ob
from oracle import schedule as osch
from paper_1708_05604_amd import synth
from tests.bruteforce import brute_force

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "dp_worked_example.json")


def test_worked_examples():
    cases = json.load(open(GOLDEN))["cases"]
    for c in cases:
        bests, bucket_of, K_eff, padded = ob.bucket_plan(c["lengths"], c["K"])
        assert list(bests) == c["bests"], c
        assert padded == c["padded"], c


def test_brute_force_matches_on_examples():
    for c in json.load(open(GOLDEN))["cases"]:
        cost, bests = brute_force(c["lengths"], c["K"])
        assert cost == c["padded"] and bests == c["bests"]


@pytest.mark.parametrize("seed", range(40))
def test_dp_equals_brute_force(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 30))
    hi = int(rng.integers(1, 25))
    lengths = rng.integers(1, hi + 1, n)
    if seed % 3 == 0:  # heavy ties
        lengths = rng.choice([3, 7, 8, 20], n)
    D = len(np.unique(lengths))
    for K in range(1, min(D, 7) + 2):
        cost, bests = brute_force(lengths, K)
        ob_bests, bucket_of, K_eff, padded = ob.bucket_plan(lengths, K)
        assert K_eff == min(K, D)
        assert padded == cost
        assert list(ob_bests) == bests, (lengths, K)


def test_invariants_on_workload_lengths():
    for name in ("tiny", "lstm2"):
        w = synth.WORKLOADS[name]
        rng = np.random.default_rng(0)
        lengths = synth.draw_lengths(rng, w.law, w.law_args, w.n)
        n, Lmax, U = len(lengths), int(lengths.max()), int(lengths.sum())
        D = len(np.unique(lengths))
        prev = None
        for K in (1, 2, 3, 5, 8):
            bests, bucket_of, K_eff, padded = ob.bucket_plan(lengths, K)
            assert bests[-1] == Lmax
            assert np.all(np.diff(bests) > 0)
            assert np.all(lengths <= bests[bucket_of])
            assert np.all((bucket_of == 0) | (lengths > bests[np.maximum(bucket_of - 1, 0)]))
            assert np.bincount(bucket_of, minlength=K_eff).sum() == n
            assert np.all(np.bincount(bucket_of, minlength=K_eff) > 0)
            assert U <= padded <= n * Lmax
            if K == 1:
                assert padded == n * Lmax
            if prev is not None:
                assert padded <= prev
            prev = padded
        if name == "tiny":
            _, _, K_eff, padded = ob.bucket_plan(lengths, D)
            assert K_eff == D and padded == U


def test_rejects_bad_input():
    with pytest.raises(ValueError):
        ob.bucket_plan([3, 0, 2], 2)
    with pytest.raises(ValueError):
        ob.bucket_plan([3, 2], 0)


def test_schedule_invariants():
    w = synth.WORKLOADS["tiny"]
    data = synth.make_workload(w, 0)
    bests, bucket_of, K_eff, _ = ob.bucket_plan(data.lengths, 2)
    keys = synth.shuffle_keys(0, 0, w.n)
    batches = osch.epoch_batches(data.lengths, bucket_of, K_eff, keys, w.batch)
    allidx = np.concatenate(batches)
    assert sorted(allidx.tolist()) == list(range(w.n))
    # buckets in ascending order, batches never straddle buckets
    bk = [set(bucket_of[b].tolist()) for b in batches]
    assert all(len(s) == 1 for s in bk)
    assert [min(s) for s in bk] == sorted(min(s) for s in bk)
    for b in batches:
        L = data.lengths[b]
        assert np.all(np.diff(L) <= 0)
        assert 1 <= len(b) <= w.batch
    # the unbucketed baseline pads more than the bucketed schedule
    _, bo1, k1, _ = ob.bucket_plan(data.lengths, 1)
    b1 = osch.epoch_batches(data.lengths, bo1, k1, keys, w.batch)
    assert osch.padded_batch_steps(data.lengths, b1) >= osch.padded_batch_steps(data.lengths, batches)


def _hand_schedule():
    # 9 sequences in 3 buckets; bucket 0 = {0, 1, 2}, 1 = {3, 4, 5, 6}, 2 = {7, 8}
    lengths = np.array([3, 2, 3, 6, 5, 6, 4, 9, 8], np.int32)
    bucket_of = np.array([0, 0, 0, 1, 1, 1, 1, 2, 2], np.int32)
    keys = np.array([2, 1, 0, 7, 5, 6, 4, 1, 0], np.uint64)
    return lengths, bucket_of, keys


def test_orderings_hand_worked():
    """Batches worked out by hand from the definitions (B = 2): inside each
    bucket the sequences go by key, pairs form the batches, each batch is
    sorted longest first."""
    lengths, bucket_of, keys = _hand_schedule()
    # bucket 0 by key: 2, 1, 0 -> pairs [2, 1], [0]; bucket 1 by key: 6, 4, 5, 3
    # -> pairs [4, 6] (4 is longer), [3, 5];
    # bucket 2 by key: 8, 7 -> sorted longest first [7, 8];
    # equal lengths (3 and 5) go by index
    asc = [[2, 1], [0], [4, 6], [3, 5], [7, 8]]
    got = osch.epoch_batches(lengths, bucket_of, 3, keys, 2)
    assert [b.tolist() for b in got] == asc
    got = osch.epoch_batches(lengths, bucket_of, 3, keys, 2, "descending")
    assert [b.tolist() for b in got] == [[7, 8], [4, 6], [3, 5], [2, 1], [0]]
    ok = np.array([9, 3, 3, 0, 0, 0, 0, 0, 0], np.uint64)  # bucket order 1, 2, 0
    got = osch.epoch_batches(lengths, bucket_of, 3, keys, 2, "random_buckets", ok)
    assert [b.tolist() for b in got] == [[4, 6], [3, 5], [7, 8], [2, 1], [0]]
    ok = np.array([4, 0, 3, 0, 1, 0, 0, 0, 0], np.uint64)  # fed: batches 1, 3, 4, 2, 0
    got = osch.epoch_batches(lengths, bucket_of, 3, keys, 2, "shuffled_batches", ok)
    assert [b.tolist() for b in got] == [[0], [3, 5], [7, 8], [4, 6], [2, 1]]


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_orderings_are_permutations_of_the_same_batches(seed):
    w = synth.WORKLOADS["tiny"]
    data = synth.make_workload(w, seed)
    _, bucket_of, K_eff, _ = ob.bucket_plan(data.lengths, 3)
    keys = synth.shuffle_keys(seed, 0, w.n)
    ok = synth.order_keys(seed, 0, w.n)
    asc = osch.epoch_batches(data.lengths, bucket_of, K_eff, keys, w.batch)
    ref = sorted(tuple(b.tolist()) for b in asc)
    for ordering in osch.ORDERINGS:
        got = osch.epoch_batches(data.lengths, bucket_of, K_eff, keys, w.batch, ordering, ok)
        assert sorted(tuple(b.tolist()) for b in got) == ref
        runs = [int(bucket_of[b[0]]) for b in got]
        if ordering == "descending":
            assert runs == sorted(runs, reverse=True)
        if ordering in ("ascending", "descending", "random_buckets"):
            # whole buckets stay together: each bucket is one contiguous run
            seen = [r for i, r in enumerate(runs) if i == 0 or runs[i - 1] != r]
            assert len(seen) == len(set(seen)) == K_eff
    # keys that rank the batches (or buckets) in their ascending order change nothing
    rising = np.arange(w.n, dtype=np.uint64)
    for ordering in ("random_buckets", "shuffled_batches"):
        got = osch.epoch_batches(data.lengths, bucket_of, K_eff, keys, w.batch, ordering, rising)
        assert [b.tolist() for b in got] == [b.tolist() for b in asc]
    falling = rising[::-1].copy()
    got = osch.epoch_batches(data.lengths, bucket_of, K_eff, keys, w.batch, "random_buckets",
                             falling)
    desc = osch.epoch_batches(data.lengths, bucket_of, K_eff, keys, w.batch, "descending")
    assert [b.tolist() for b in got] == [b.tolist() for b in desc]
    got = osch.epoch_batches(data.lengths, bucket_of, K_eff, keys, w.batch, "shuffled_batches",
                             falling)
    assert [b.tolist() for b in got] == [b.tolist() for b in asc[::-1]]
    with pytest.raises(ValueError):
        osch.epoch_batches(data.lengths, bucket_of, K_eff, keys, w.batch, "sideways")
