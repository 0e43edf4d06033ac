"""The float64 oracle over whole mini-batches, split across worker processes.

Test infrastructure only (see oracle/__init__.py): the GPU-parity tests use it
on batches too long for one process, the benchmark for its CPU baseline on
all host cores.  Workers import only this package and numpy (never the GPU
path) and run with one BLAS thread each.

Sequences are independent and the per-frame loss and its gradient are means
over the batch's valid frames, so a batch split into parts of N_p frames
gives loss = sum_p (N_p / N) loss_p, and the same weights for the gradient --
the batch-split invariance the oracle's tests pin.  A batch's sequences are
dealt longest first, each to the least loaded part; each part is one task
that returns its N_p-weighted sums, and the parent adds them.
"""
from __future__ import annotations

import concurrent.futures
import multiprocessing
import os
import time

import numpy as np

from oracle import rnn as orn


def _work(model_args, theta, xs, ys, need_tops):
    t0 = time.perf_counter()
    m = orn.Model(*model_args)
    n_part = sum(len(y) for y in ys)
    loss, grad, tops = orn.forward_backward(m, np.asarray(theta, np.float64), xs, ys)
    tops = [np.asarray(t, np.float32) for t in tops] if need_tops else None
    return n_part, loss * n_part, grad * n_part, tops, time.perf_counter() - t0


def _worker_init(nice):
    if nice > 0:
        os.nice(nice)
    from threadpoolctl import threadpool_limits
    threadpool_limits(limits=1)  # also set by the environment at start


def _ready():
    return os.getpid()


def default_workers() -> int:
    """The CPUs this process may run on, at most 16 (a host that shares its
    cores between several GPUs gives one GPU's process about that many,
    whatever it reports)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


class Pool:
    """Worker processes (started fresh, not forked) shared by any number of
    batches; submit() returns a BatchJob whose result() waits for it."""

    def __init__(self, workers: int | None = None, nice: int = 0):
        """nice > 0 lowers the workers' scheduling priority (work running
        beside them in the parent keeps precedence)."""
        self.workers = default_workers() if workers is None else max(1, int(workers))
        # One BLAS thread per worker (the work is split by processes).
        env = {"OMP_NUM_THREADS": "1", "OPENBLAS_NUM_THREADS": "1"}
        saved = {k: os.environ.get(k) for k in env}
        os.environ.update(env)
        try:
            self.ex = concurrent.futures.ProcessPoolExecutor(
                max_workers=self.workers, mp_context=multiprocessing.get_context("spawn"),
                initializer=_worker_init, initargs=(nice,))
            # The workers start on demand: start them all now, while the
            # environment above is in place.
            for f in [self.ex.submit(_ready) for _ in range(self.workers)]:
                f.result()
        finally:
            for k, v in saved.items():
                if v is None:
                    os.environ.pop(k, None)
                else:
                    os.environ[k] = v

    def submit(self, model: "orn.Model", theta, data, order, parts: int | None = None,
               need_tops: bool = True, label: str = "") -> "BatchJob":
        """Oracle loss, gradient and top-layer outputs of the batch made of
        sequences `order` of `data` (synth.Data) under parameters `theta`
        (float32 or float64; sent to the workers in that type)."""
        return BatchJob(self, model, theta, data, order,
                        self.workers if parts is None else parts, need_tops, label)

    def close(self, kill: bool = False):
        """Stops the workers; kill=True ends running tasks too."""
        if kill:
            for p in list(getattr(self.ex, "_processes", {}).values()):
                p.terminate()
        self.ex.shutdown(wait=not kill, cancel_futures=True)


class BatchJob:
    def __init__(self, pool, model, theta, data, order, parts, need_tops, label):
        self.label = label
        self.order = [int(s) for s in order]
        lens = [int(data.lengths[s]) for s in self.order]
        self.n_valid = sum(lens)
        w = max(1, min(parts, len(self.order)))
        groups = [[] for _ in range(w)]
        load = [0] * w
        for b in sorted(range(len(self.order)), key=lambda b: -lens[b]):
            p = int(np.argmin(load))
            groups[p].append(b)
            load[p] += lens[b]
        self.groups = [sorted(g) for g in groups if g]
        args = (model.cell, model.num_layers, model.bidirectional, model.input_dim, model.hidden,
                model.num_classes)
        theta = np.asarray(theta)
        if theta.dtype != np.float32:
            theta = theta.astype(np.float64)
        self.t0 = time.perf_counter()
        self.futures = []
        for rows in self.groups:
            seqs = [self.order[b] for b in rows]
            xs = [data.X[data.offsets[s]:data.offsets[s + 1]] for s in seqs]
            ys = [data.Y[data.offsets[s]:data.offsets[s + 1]] for s in seqs]
            self.futures.append(pool.ex.submit(_work, args, theta, xs, ys, need_tops))

    def result(self, log=None):
        """(loss, grad float64, tops: per batch row a float32 [L, H_top] array
        or None)."""
        loss, grad = 0.0, None
        tops = [None] * len(self.order)
        index = {f: i for i, f in enumerate(self.futures)}
        for k, fut in enumerate(concurrent.futures.as_completed(self.futures)):
            i = index[fut]
            n_part, l_sum, g_sum, t_list, secs = fut.result()
            if log:
                log(f"[oracle] {self.label}: part {i} ({n_part} frames) {secs:.1f} s "
                    f"({k + 1}/{len(self.futures)} done, {time.perf_counter() - self.t0:.1f} s)")
            loss += l_sum
            grad = g_sum if grad is None else grad + g_sum
            if t_list is not None:
                for b, t in zip(self.groups[i], t_list):
                    tops[b] = t
        return loss / self.n_valid, grad / self.n_valid, tops
