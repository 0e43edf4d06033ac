"""Host-side checks of librnnbkt.so that need no GPU: the library loads and
exports every entry point of include/rnnbkt.h; the planner and the epoch
schedule match the oracle bit for bit; argument validation rejects bad
input before touching the GPU."""
import os
import re

import numpy as np
import pytest

from oracle import bucketing as ob
from oracle import rnn as orn
from oracle import schedule as osch
from paper_1708_05604_amd import lib, synth
from tests.bruteforce import brute_force

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_exports_every_declared_symbol():
    header = open(os.path.join(ROOT, "include", "rnnbkt.h")).read()
    declared = set(re.findall(r"\b(rnnbkt_[a-z_]+)\s*\(", header))
    assert declared, "no declarations found"
    assert declared == set(lib.exported_symbols())
    L = lib.load()
    for name in declared:
        assert hasattr(L, name), name
    assert "gfx950" in lib.version()


@pytest.mark.parametrize("seed", range(30))
def test_planner_matches_brute_force(seed):
    rng = np.random.default_rng(1000 + seed)
    n = int(rng.integers(1, 40))
    lengths = rng.integers(1, int(rng.integers(2, 30)), n)
    if seed % 4 == 0:
        lengths = rng.choice([2, 5, 6, 11], n)
    D = len(np.unique(lengths))
    for K in range(1, D + 3):
        cost, bests = brute_force(lengths, K)
        up, bof, keff, padded = lib.bucket_plan(lengths, K)
        assert keff == min(K, D)
        assert padded == cost
        assert list(up) == bests


@pytest.mark.parametrize("name", list(synth.WORKLOADS))
def test_planner_matches_oracle_on_workloads(name):
    w = synth.WORKLOADS[name]
    lengths = synth.draw_lengths(np.random.default_rng(0), w.law, w.law_args, w.n)
    for K in sorted(set(w.k_list) | {2, 3}):
        if name == "longtail" and K == 32:
            continue  # covered by the slow test below
        a = ob.bucket_plan(lengths, K)
        b = lib.bucket_plan(lengths, K)
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
        assert a[2] == b[2] and a[3] == b[3]


@pytest.mark.slow
def test_planner_matches_oracle_longtail_32():
    w = synth.WORKLOADS["longtail"]
    lengths = synth.draw_lengths(np.random.default_rng(0), w.law, w.law_args, w.n)
    a = ob.bucket_plan(lengths, 32)
    b = lib.bucket_plan(lengths, 32)
    assert np.array_equal(a[0], b[0]) and a[3] == b[3]


def test_planner_edge_cases():
    assert lib.bucket_plan([7], 1)[3] == 7
    up, bof, keff, padded = lib.bucket_plan([7], 5)
    assert keff == 1 and list(up) == [7] and padded == 7
    up, bof, keff, padded = lib.bucket_plan([3] * 100, 4)
    assert keff == 1 and padded == 300
    big = np.full(10, 2_000_000_000 // 10, np.int32)
    assert lib.bucket_plan(big, 1)[3] == int(big.sum())
    # The histogram covers the distinct lengths only: a length at the int32
    # limit costs no memory proportional to it; costs are summed in int64.
    top = np.iinfo(np.int32).max
    up, bof, keff, padded = lib.bucket_plan(np.array([top, 1, 5, top], np.int32), 2)
    assert keff == 2 and list(up) == [5, top] and list(bof) == [1, 0, 0, 1]
    assert padded == 2 * 5 + 2 * top
    with pytest.raises(lib.RnnbktError) as e:
        lib.bucket_plan([1, 0, 2], 2)
    assert e.value.code == lib.EINVAL
    with pytest.raises(lib.RnnbktError):
        lib.bucket_plan([1, 2], 0)
    with pytest.raises(lib.RnnbktError):
        lib.bucket_plan([], 1)


@pytest.mark.parametrize("name,K", [("tiny", 1), ("tiny", 2), ("lstm2", 8), ("longtail", 4)])
def test_schedule_matches_oracle(name, K):
    w = synth.WORKLOADS[name]
    lengths = synth.draw_lengths(np.random.default_rng(0), w.law, w.law_args, w.n)
    _, bof, keff, _ = lib.bucket_plan(lengths, K)
    for epoch in (0, 1):
        keys = synth.shuffle_keys(0, epoch, w.n)
        a = osch.epoch_batches(lengths, bof, keff, keys, w.batch)
        b = lib.epoch_schedule(lengths, bof, keff, keys, w.batch)
        assert len(a) == len(b)
        for x, y in zip(a, b):
            assert np.array_equal(x, y)


def test_schedule_ties_and_partial_batches():
    lengths = np.array([4, 4, 4, 1, 1, 9, 9], np.int32)
    keys = np.array([5, 5, 1, 3, 3, 0, 2], np.uint64)  # equal keys fall back to index
    bof = np.zeros(7, np.int32)
    a = osch.epoch_batches(lengths, bof, 1, keys, 3)
    b = lib.epoch_schedule(lengths, bof, 1, keys, 3)
    assert [x.tolist() for x in a] == [x.tolist() for x in b]
    assert [len(x) for x in b] == [3, 3, 1]


def _desc(w):
    return lib.ModelDesc.of(w.cell, w.num_layers, w.input_dim, w.hidden, w.num_classes,
                            w.bidirectional, w.gemm_dtype)


@pytest.mark.parametrize("name", list(synth.WORKLOADS))
def test_param_count_matches_oracle(name):
    w = synth.WORKLOADS[name]
    m = orn.Model(w.cell, w.num_layers, w.bidirectional, w.input_dim, w.hidden, w.num_classes)
    assert lib.param_count(_desc(w)) == orn.param_count(m)


def test_buffer_sizes_monotone():
    w = synth.WORKLOADS["bilstm3"]
    d = _desc(w)
    base = lib.buffer_sizes(d, 100, 8, 400)
    for args in ((101, 8, 400), (100, 9, 400), (100, 8, 401), (200, 16, 3000)):
        r, ws = lib.buffer_sizes(d, *args)
        assert r >= base[0] and ws >= base[1]
    assert lib.buffer_sizes(d, 100, 8, 400) == base


def test_validation_errors_before_launch():
    w = synth.WORKLOADS["tiny"]
    d = _desc(w)
    bad = lib.ModelDesc.of(0, 1, 4, 33, 20, 0, 0)
    with pytest.raises(lib.RnnbktError) as e:
        lib.param_count(bad)
    assert e.value.code == lib.EUNSUPPORTED
    with pytest.raises(lib.RnnbktError) as e:
        lib.param_count(lib.ModelDesc.of(3, 1, 4, 32, 20, 0, 0))
    assert e.value.code == lib.EINVAL
    L = lib.load()
    import ctypes
    lens = np.array([5, 6], np.int32)  # not non-increasing
    rc = L.rnnbkt_lstm_fwd(ctypes.byref(d), 16, 16, 16, lens.ctypes.data_as(lib._i32p), 5, 2,
                           16, 1 << 30, 16, 1 << 30, 16, None)
    assert rc == lib.EINVAL and "non-increasing" in lib.last_error()
    lens = np.array([6, 5], np.int32)
    rc = L.rnnbkt_lstm_fwd(ctypes.byref(d), 16, 16, 16, lens.ctypes.data_as(lib._i32p), 7, 2,
                           16, 1 << 30, 16, 1 << 30, 16, None)
    assert rc == lib.EINVAL and "T_max" in lib.last_error()
    rc = L.rnnbkt_lstm_fwd(ctypes.byref(d), None, 16, 16, lens.ctypes.data_as(lib._i32p), 6, 2,
                           16, 1 << 30, 16, 1 << 30, 16, None)
    assert rc == lib.EINVAL
    rc = L.rnnbkt_lstm_fwd(ctypes.byref(d), 16, 16, 16, lens.ctypes.data_as(lib._i32p), 6, 2,
                           16, 10, 16, 10, 16, None)
    assert rc == lib.EINVAL and "too small" in lib.last_error()
    rc = L.rnnbkt_lstm_bwd(ctypes.byref(d), 16, lens.ctypes.data_as(lib._i32p), 6, 2,
                           16, 10, 16, 10, 16, None)
    assert rc == lib.EINVAL
    rc = L.rnnbkt_sgd_apply(None, 16, 10, 0.1, None)
    assert rc == lib.EINVAL
    rc = L.rnnbkt_sgd_apply(18, 16, 10, 0.1, None)
    assert rc == lib.EINVAL and "aligned" in lib.last_error()
    rc = L.rnnbkt_adadelta_apply(16, 16, None, 16, 10, 0.95, 1e-6, 1.0, None)
    assert rc == lib.EINVAL and "null" in lib.last_error()
    rc = L.rnnbkt_adadelta_apply(16, 16, 16, 20, 10, 0.95, 1e-6, 1.0, None)
    assert rc == lib.EINVAL and "aligned" in lib.last_error()
    for rho, eps, lr in ((1.0, 1e-6, 1.0), (-0.1, 1e-6, 1.0), (0.95, 0.0, 1.0), (0.95, 1e-6, 0.0)):
        rc = L.rnnbkt_adadelta_apply(16, 16, 16, 16, 10, rho, eps, lr, None)
        assert rc == lib.EINVAL, (rho, eps, lr)
    assert L.rnnbkt_adadelta_apply(16, 16, 16, 16, -1, 0.95, 1e-6, 1.0, None) == lib.EINVAL
    assert L.rnnbkt_adadelta_apply(16, 16, 16, 16, 0, 0.95, 1e-6, 1.0, None) == lib.OK


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(lib, "_lib", None)
    monkeypatch.setattr(lib, "LIB_PATH", str(tmp_path / "absent.so"))
    with pytest.raises(lib.LibraryMissing):
        lib.load()
    with pytest.raises(lib.LibraryMissing):
        lib.bucket_plan([1, 2], 1)


@pytest.mark.parametrize("ordering", ["ascending", "descending", "random_buckets",
                                      "shuffled_batches"])
@pytest.mark.parametrize("name,K", [("tiny", 3), ("lstm2", 8), ("longtail", 1)])
def test_ordered_schedule_matches_oracle(ordering, name, K):
    w = synth.WORKLOADS[name]
    lengths = synth.draw_lengths(np.random.default_rng(1), w.law, w.law_args, w.n)
    _, bof, keff, _ = lib.bucket_plan(lengths, K)
    for epoch in (0, 1):
        keys = synth.shuffle_keys(1, epoch, w.n)
        ok = synth.order_keys(1, epoch, w.n)
        a = osch.epoch_batches(lengths, bof, keff, keys, w.batch, ordering, ok)
        b = lib.epoch_schedule(lengths, bof, keff, keys, w.batch, ordering, ok)
        assert len(a) == len(b)
        for x, y in zip(a, b):
            assert np.array_equal(x, y)


def test_ordered_schedule_rejects_bad_input():
    lengths = np.array([3, 1, 2], np.int32)
    bof = np.zeros(3, np.int32)
    keys = np.arange(3, dtype=np.uint64)
    with pytest.raises(lib.RnnbktError):
        lib.epoch_schedule(lengths, bof, 1, keys, 2, "random_buckets")  # needs order_keys
    with pytest.raises(lib.RnnbktError):
        lib.epoch_schedule(lengths, bof, 1, keys, 2, "shuffled_batches", np.zeros(2, np.uint64))
    with pytest.raises(lib.RnnbktError):
        lib.epoch_schedule(lengths, bof, 1, keys, 2, "sideways")
    # descending needs no keys and equals the ascending list for one bucket
    a = lib.epoch_schedule(lengths, bof, 1, keys, 2, "descending")
    b = lib.epoch_schedule(lengths, bof, 1, keys, 2)
    assert [x.tolist() for x in a] == [x.tolist() for x in b]


def test_epoch_aggregate_validation():
    """Bad arguments are rejected before any launch (host addresses only)."""
    L = lib.load()
    base, prev = 1 << 20, 1 << 30

    def call(reps=base, R=2, stride=8, n=8, pv=prev, beta=1e-6):
        return L.rnnbkt_epoch_aggregate(reps, R, stride, n, pv, beta, None)

    assert call(reps=None) == lib.EINVAL
    assert call(pv=None) == lib.EINVAL
    assert call(R=0) == lib.EINVAL
    assert call(R=1025) == lib.EINVAL
    assert call(n=-1) == lib.EINVAL
    assert call(stride=6, n=6) == lib.EINVAL          # stride not a multiple of 4
    assert call(stride=4, n=8) == lib.EINVAL          # stride < n
    assert call(reps=base + 4) == lib.EINVAL          # misaligned
    assert call(beta=float("nan")) == lib.EINVAL
    assert call(pv=base + 4 * 8) == lib.EINVAL        # prev overlaps replica 1
    assert call(pv=base + 4 * 4) == lib.EINVAL        # prev overlaps replica 0's tail
    assert call(n=0) == lib.OK                        # nothing to do, nothing launched


def test_set_concurrency_validation():
    L = lib.load()
    assert L.rnnbkt_set_concurrency(0) == lib.EINVAL
    assert L.rnnbkt_set_concurrency(65) == lib.EINVAL
    assert L.rnnbkt_set_concurrency(3) == lib.OK
    assert L.rnnbkt_set_concurrency(1) == lib.OK
