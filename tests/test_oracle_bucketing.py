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


@pytest.mark.parametrize("seed", range(10))
def test_loop_form_equals_vector_form(seed):
    rng = np.random.default_rng(100 + seed)
    lengths = rng.integers(1, 40, int(rng.integers(1, 60)))
    f = ob.length_histogram(lengths)
    D = int(np.count_nonzero(f))
    for Q in range(1, D + 1):
        a = ob.dynamic_bucketing_loops(Q, f)
        b = ob.dynamic_bucketing(Q, f)
        assert a[0] == b[0] and a[1] == b[1]


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
