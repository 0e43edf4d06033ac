"""Oracle references of the long-batch GPU tests, computed in the background.

The session hook in conftest.py starts them when the tests are selected,
before any test touches the GPU, on one pool of worker processes shared by
all cases (oracle/pool.py); the tests collect them after their GPU run.  The
batches are chosen with the oracle's own planner and schedule; the tests
check that the library picks the same ones.
"""
from __future__ import annotations

import sys

import numpy as np

from oracle import bucketing as ob
from oracle import pool as opool
from oracle import rnn as orn
from oracle import schedule as osch
from paper_1708_05604_amd import synth

# (workload, K, T_max, B, N) of the batch holding the longest sequence of
# epoch 0 (ties: the most frames); the sizes are checked so that a change of
# the generators or the planner cannot silently swap in a shorter batch.
CASES = [
    ("bilstm3", 16, 2500, 64, 144629),
    ("longtail", 16, 4000, 24, 87769),
    ("longtail", 1, 4000, 128, 23650),
    ("gru2", 8, 1500, 96, 118323),
    ("lstm2p", 8, 1500, 64, 78768),
]


def case_id(name, K):
    return f"{name}-K{K}"


BY_ID = {case_id(c[0], c[1]): c for c in CASES}

_pool = None
_blas_limit = None
_jobs = {}


def model_of(w: synth.Workload) -> orn.Model:
    return orn.Model(w.cell, w.num_layers, w.bidirectional, w.input_dim, w.hidden,
                     w.num_classes)


def longest_batch(name: str, K: int, epoch: int = 0):
    """(workload data, batch order) by the oracle's planner and schedule."""
    w = synth.WORKLOADS[name]
    data = synth.make_workload(w, 0, param_count=orn.param_count(model_of(w)))
    _, bof, keff, _ = ob.bucket_plan(data.lengths, K)
    batches = osch.epoch_batches(data.lengths, bof, keff, synth.shuffle_keys(0, epoch, w.n),
                                 w.batch)
    order = max(batches, key=lambda bt: (int(data.lengths[bt].max()), int(data.lengths[bt].sum())))
    return data, np.asarray(order, np.int64)


def _log(msg):
    print(msg, file=sys.stderr, flush=True)


def start(ids):
    """Submits the oracle work of the given case ids (idempotent).  Every
    batch is chosen before the first is submitted: the workers would
    otherwise compete with the planning for the CPUs."""
    global _pool
    todo = [cid for cid in dict.fromkeys(ids) if cid not in _jobs]
    if not todo:
        return
    chosen = [(cid, longest_batch(*BY_ID[cid][:2])) for cid in todo]
    if _pool is None:
        # Four CPUs stay with the rest of the suite, which runs meanwhile
        # (and has oracle work of its own): the workers get a lower priority,
        # and BLAS in this process is held to four threads while they run.
        global _blas_limit
        free = 4
        _pool = opool.Pool(max(1, opool.default_workers() - free), nice=10)
        from threadpoolctl import threadpool_limits
        _blas_limit = threadpool_limits(limits=free)
    for cid, (data, order) in chosen:
        w = synth.WORKLOADS[BY_ID[cid][0]]
        _jobs[cid] = (data, order,
                      _pool.submit(model_of(w), data.params, data, order, label=cid))
        _log(f"[oracle] {cid}: {len(order)} sequences, {int(data.lengths[order].sum())} frames "
             f"submitted to {_pool.workers} workers")


def get(cid):
    """(data, order, BatchJob) of a case, submitting it now if needed."""
    start([cid])
    return _jobs[cid]


def stop():
    global _pool, _blas_limit
    if _pool is not None:
        _pool.close(kill=True)
        _pool = None
    if _blas_limit is not None:
        _blas_limit.restore_original_limits()
        _blas_limit = None
    _jobs.clear()
