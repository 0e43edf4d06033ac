"""Throughput of bucketed LSTM training on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload bilstm3] [--K 16]

A step is one epoch: every mini-batch of the epoch schedule, in the paper's
order (buckets shortest first, Sec. IV.A), through the whole hot path --
rnnbkt_lstm_fwd (packing, input projections, recurrent steps, output layer,
softmax cross-entropy), rnnbkt_lstm_bwd (output-layer gradients,
backpropagation through time, weight gradients) and rnnbkt_sgd_apply.  The
timed steps replay the schedule of epoch 0 (shuffle keys of epoch 0), whose
batches are all staged in device memory before timing.  The bucket plan and
the schedule run once on the host before timing (they depend only on the
lengths) and are timed separately.  The default workload is the largest
one, a 3-layer bidirectional LSTM at K = 16 buckets.

Printed: one JSON line with the metric (useful, i.e. non-pad, timesteps per
second of fwd+bwd+update over whole epochs), one whole epoch at K=1 (the
unbucketed baseline, random batches), pad-waste counts, the fraction of the
matrix-core peak, the roofline entry of the kernel class that takes the most
GPU time (HIP events in a second pass over one epoch), HBM rates of the
streaming kernels, and the float64 oracle timed on a bounded sample of the
same workload on the host cores (all of them, and one thread).
"""
from __future__ import annotations

import argparse
import collections
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_1708_05604_amd import lib, synth  # noqa: E402

METRIC = "useful (non-pad) LSTM timesteps/sec fwd+bwd on 1 GPU; MFMA util %; pad waste %"
PEAK_TFLOPS = {synth.FP32: 157.3, synth.BF16: 2500.0}
PEAK_HBM_GBS = 8000.0
ROOT = os.path.dirname(os.path.abspath(__file__))
# Kernel sources whose hash keys the recorded byte counters: after any change
# to them the counters no longer describe the kernel and traffic is null.
TRAFFIC_SOURCES = ("paper_1708_05604_amd/csrc/rnn_persistent.hip", "paper_1708_05604_amd/csrc/kernels.h")


def recorded_traffic(workload, K, kind):
    """HBM bytes per launch of the dominant kernel from the rocprofv3 FETCH_SIZE /
    WRITE_SIZE runs summarised under profiles/, or None when no record matches
    this workload, kernel and the current kernel sources."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"{workload}_k{K}_traffic.txt")
    if not os.path.exists(path):
        return None
    rec = {}
    for line in open(path):
        if "=" in line and not line.lstrip().startswith("#"):
            k, v = line.split("=", 1)
            rec[k.strip()] = v.strip()
    h = hashlib.sha256()
    for src in TRAFFIC_SOURCES:
        with open(os.path.join(ROOT, src), "rb") as f:
            h.update(f.read())
    if rec.get("kernel_kind") != kind or rec.get("sources_sha256_16") != h.hexdigest()[:16]:
        return None
    return float(rec["fetch_bytes_per_launch"]) + float(rec["write_bytes_per_launch"])
TILE_M = 16


def flops_per_useful_step(w: synth.Workload) -> int:
    """Matrix-core flops per valid frame of one training step (input and
    recurrent products forward, the same products and the weight gradients
    backward, output layer forward and backward)."""
    G = 3 if w.cell == synth.GRU else 4
    H, dirs = w.hidden, 2 if w.bidirectional else 1
    GH = G * H
    total = 0
    for layer in range(w.num_layers):
        din = w.input_dim if layer == 0 else dirs * H
        fwd = 2 * GH * (din + H)
        bwd = 2 * GH * din * (2 if layer > 0 else 1) + 4 * GH * H
        total += dirs * (fwd + bwd)
    total += 6 * dirs * H * w.num_classes
    return total


def param_count(w: synth.Workload) -> int:
    """Length of the flat parameter vector (the layout of include/rnnbkt.h);
    checked against rnnbkt_param_count once the library is loaded."""
    G = 3 if w.cell == synth.GRU else 4
    H, dirs = w.hidden, 2 if w.bidirectional else 1
    total = 0
    for layer in range(w.num_layers):
        din = w.input_dim if layer == 0 else dirs * H
        per = G * H * (din + H) + G * H * (2 if w.cell == synth.GRU else 1)
        if w.cell == synth.LSTM_PEEPHOLE:
            per += 3 * H
        total += dirs * per
    return total + w.num_classes * (dirs * H + 1)


def describe(w: synth.Workload, K: int, seed: int = 0) -> str:
    cell = {synth.LSTM: "LSTM", synth.GRU: "GRU", synth.LSTM_PEEPHOLE: "peephole LSTM"}[w.cell]
    bi = "bidirectional " if w.bidirectional else ""
    return (f"{w.name}: {w.num_layers}-layer {bi}{cell} D={w.input_dim} H={w.hidden} "
            f"C={w.num_classes}, {w.n} sequences {w.law}{w.law_args}, B={w.batch}, K={K}, "
            f"{'bf16' if w.gemm_dtype == synth.BF16 else 'fp32'} GEMMs, seed {seed}")


class Epoch:
    """One epoch's batches staged on the GPU."""

    def __init__(self, w, data, K, epoch, torch, dev, targets=None, ordering="ascending",
                 seed=0):
        t0 = time.perf_counter()
        self.upper, bof, self.keff, self.p_bucket = lib.bucket_plan(data.lengths, K)
        self.plan_ms = (time.perf_counter() - t0) * 1e3
        t0 = time.perf_counter()
        self.batches = lib.epoch_schedule(data.lengths, bof, self.keff,
                                          synth.shuffle_keys(seed, epoch, w.n), w.batch,
                                          ordering, synth.order_keys(seed, epoch, w.n))
        self.sched_ms = (time.perf_counter() - t0) * 1e3
        self.lens, self.x, self.y, self.useful = [], [], [], []
        self.p_batch = 0
        self.p_exec = 0
        for order in self.batches:
            x, y, L = synth.padded_batch(data, order)
            self.lens.append(L)
            self.x.append(torch.from_numpy(x).to(dev))
            self.y.append(torch.from_numpy(y).to(dev))
            self.useful.append(int(L.sum()))
            self.p_batch += len(L) * int(L[0])
            bt = np.bincount(L, minlength=int(L[0]) + 1)[::-1].cumsum()[::-1][1:]
            self.p_exec += int(np.sum((bt + TILE_M - 1) // TILE_M * TILE_M))
        # CTC label strings per batch ([B, U_max] device tensor, host lengths)
        self.tg, self.tl = [], []
        if targets is not None:
            for order in self.batches:
                tl = np.array([len(targets[s]) for s in order], np.int32)
                tm = np.zeros((len(order), int(tl.max())), np.int32)
                for b, s in enumerate(order):
                    tm[b, :tl[b]] = targets[s]
                self.tg.append(torch.from_numpy(tm).to(dev))
                self.tl.append(tl)
        self.max_U = max((int(t.max()) for t in self.tl), default=0)
        self.U = int(sum(self.useful))
        self.max_T = max(int(L[0]) for L in self.lens)
        self.max_B = max(len(L) for L in self.lens)
        self.max_N = max(self.useful)


# The host runs at most this many training steps ahead of the GPU: an epoch
# of bilstm3 enqueues about 13,000 launches, and with no bound the runtime's
# queues fill up and the host blocks inside launch calls; an epoch then took
# 1912-1960 ms from run to run, against 1912-1913 ms paced (16 steps ahead:
# about 0.1 s of work, so the GPU never waits for the host).
PACE_STEPS = 16


def run_steps(ep, state, first, count, torch):
    desc, params, grads, reserve, workspace, loss, lr, opt, ctc_ws = state
    useful = 0
    nb = len(ep.batches)
    marks = collections.deque()
    for k in range(count):
        i = (first + k) % nb
        if ctc_ws is None:
            lib.lstm_fwd(desc, params, ep.x[i], ep.y[i], ep.lens[i], reserve, workspace, loss)
        else:
            lib.lstm_fwd_ctc(desc, params, ep.x[i], ep.tg[i], ep.tl[i], ep.lens[i], reserve,
                             workspace, ctc_ws, loss)
        lib.lstm_bwd(desc, params, ep.lens[i], reserve, workspace, grads)
        if opt is None:
            lib.sgd_apply(params, grads, lr)
        else:
            lib.adadelta_apply(params, grads, opt[0], opt[1])
        useful += ep.useful[i]
        mark = torch.cuda.Event()
        mark.record()
        marks.append(mark)
        if len(marks) > PACE_STEPS:
            marks.popleft().synchronize()
    return useful


def timed_epochs(ep, state, warmup, steps, torch):
    """`warmup` untimed epochs, then `steps` epochs back to back with an
    event between epochs (inside the timed region the host only waits for
    steps PACE_STEPS behind the one it enqueues), device synchronised on both
    sides.  Returns the seconds of each epoch."""
    nb = len(ep.batches)
    for _ in range(warmup):
        run_steps(ep, state, 0, nb, torch)
    torch.cuda.synchronize()
    lib.sync_check()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    ev[0].record()
    for i in range(steps):
        run_steps(ep, state, 0, nb, torch)
        ev[i + 1].record()
    torch.cuda.synchronize()
    lib.sync_check()
    return [ev[i].elapsed_time(ev[i + 1]) / 1e3 for i in range(steps)]


class Replicated:
    """R training replicas on R streams of the one GPU, the paper's parallel
    scheme (Sec. III.B) with a portion of the epoch per replica: replica r
    takes the epoch's batches r, r + R, ...; at the epoch end eq. 3 merges
    them (rnnbkt_epoch_aggregate) and every replica continues from the
    merged parameters."""

    def __init__(self, R, desc, data, rb, wb, lr, optimizer, ctc_bytes, torch, dev):
        self.torch = torch
        P = len(data.params)
        self.P = P
        stride = (P + 3) // 4 * 4
        self.reps = torch.zeros((R, stride), dtype=torch.float32, device=dev)
        init = torch.from_numpy(data.params).to(dev)
        for r in range(R):
            self.reps[r, :P] = init
        self.prev = init.clone()
        self.states = []
        for r in range(R):
            g = torch.zeros(P, dtype=torch.float32, device=dev)
            opt = None
            if optimizer == "adadelta":
                opt = (torch.zeros_like(g), torch.zeros_like(g))
            cw = None if ctc_bytes is None else torch.empty(ctc_bytes, dtype=torch.uint8,
                                                            device=dev)
            self.states.append((desc, self.reps[r, :P], g,
                                torch.empty(rb, dtype=torch.uint8, device=dev),
                                torch.empty(wb, dtype=torch.uint8, device=dev),
                                torch.zeros(1, dtype=torch.float32, device=dev), lr, opt, cw))
        self.streams = [torch.cuda.Stream() for _ in range(R)]
        torch.cuda.synchronize()

    def run(self, ep, first, count):
        useful = 0
        nb = len(ep.batches)
        R = len(self.streams)
        for k in range(count):
            with self.torch.cuda.stream(self.streams[k % R]):
                useful += run_steps(ep, self.states[k % R], (first + k) % nb, 1, self.torch)
        return useful

    def merge(self):
        cur = self.torch.cuda.current_stream()
        for s in self.streams:
            cur.wait_stream(s)
        lib.epoch_aggregate(self.reps, self.prev, n=self.P)
        for s in self.streams:
            s.wait_stream(cur)


def timed_replicated(ep, rep, warmup, steps, torch):
    """One epoch portion per replica, concurrently, then the eq. 3 merge;
    host clock around it with the device synchronised on both sides."""
    rep.run(ep, 0, warmup)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    useful = rep.run(ep, warmup, steps)
    rep.merge()
    torch.cuda.synchronize()
    secs = time.perf_counter() - t0
    lib.sync_check()
    return useful, secs


def latency_floor(w, ep, state, kinds, torch, dev, reps=3):
    """Latency floor of the recurrences: (sequential step phases of the epoch)
    x (minimum time per step at M = B).  The minimum is measured on the same
    resident kernels over a batch of B sequences that all have the epoch's
    longest length (capped by the staged buffers), where no row group ever
    idles and the launch prologue is spread over the most steps; the phases
    are the epoch's launches per batch times each batch's step count.
    floor_frac = floor / measured recurrence time of the epoch."""
    desc, params, grads, reserve, workspace, loss = state[:6]
    nb = len(ep.batches)
    B = w.batch
    T0 = min(ep.max_T, ep.max_N // B)
    gen = torch.Generator().manual_seed(1)
    x = (0.5 * torch.randn(T0, B, w.input_dim, generator=gen)).to(dev)
    y = torch.randint(0, w.num_classes, (T0, B), generator=gen, dtype=torch.int32).to(dev)
    L = np.full(B, T0, np.int32)
    g2 = torch.zeros_like(grads)

    def once():
        lib.lstm_fwd(desc, params, x, y, L, reserve, workspace, loss)
        lib.lstm_bwd(desc, params, L, reserve, workspace, g2)

    once()
    torch.cuda.synchronize()
    lib.kernel_timer(True)
    for _ in range(reps):
        once()
    torch.cuda.synchronize()
    lib.kernel_timer(False)
    lib.sync_check()
    t_sum = sum(int(Lb[0]) for Lb in ep.lens)
    out = {"uniform_batch": {"B": B, "T": T0, "reps": reps}}
    for kind in ("fwd", "bwd"):
        u = lib.kernel_timer_read("step_" + kind)
        per_call = max(1, round(u["launches"] / reps))
        t_min_us = 1e3 * u["ms"] / (reps * T0 * per_call)
        per_batch = max(1, round(kinds["step_" + kind]["launches"] / nb))
        phases = per_batch * t_sum
        floor_ms = phases * t_min_us / 1e3
        measured_ms = kinds["step_" + kind]["ms"]
        out[kind] = {"min_us_per_step": t_min_us, "launches_per_batch": per_batch,
                     "step_phases": phases, "floor_ms": floor_ms, "measured_ms": measured_ms,
                     "floor_frac": floor_ms / measured_ms}
    return out


def cpu_sample(w, data, K):
    """The oracle baseline's fixed batch order: the first batch of every
    bucket of epoch 0 (shortest bucket first), then the batch holding the
    longest sequence -- chosen with the oracle's own planner and schedule."""
    from oracle import bucketing as ob
    from oracle import schedule as osch
    _, bof, keff, _ = ob.bucket_plan(data.lengths, K)
    batches = osch.epoch_batches(data.lengths, bof, keff, synth.shuffle_keys(0, 0, w.n), w.batch)
    out, seen = [], set()
    for order in batches:
        b = int(bof[order[0]])
        if b not in seen:
            seen.add(b)
            out.append((f"bucket {b}", order))
    longest = max(batches, key=lambda bt: (int(data.lengths[bt].max()), int(data.lengths[bt].sum())))
    out.append(("longest", longest))
    return out


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown CPU"


def cpu_baseline(w, data, K, lr, budget_s=12.0):
    """The float64 oracle on the host cores, training: fwd+bwd of each batch
    of cpu_sample() in turn, the SGD step carried into the next batch, until
    about `budget_s` seconds of work.  Twice: on every CPU this process may
    use (the batch's sequences split over worker processes with one BLAS
    thread each, at most 16), and on one thread.  The first figure is the
    reported baseline; the second is given beside it."""
    from threadpoolctl import threadpool_limits

    from oracle import pool as opool
    from oracle import rnn as orn
    m = orn.Model(w.cell, w.num_layers, w.bidirectional, w.input_dim, w.hidden, w.num_classes)
    sample = cpu_sample(w, data, K)

    def train(step, max_batches=None):
        theta = data.params.astype(np.float64)
        used, useful, t_total = [], 0, 0.0
        for name, order in sample[:max_batches]:
            t0 = time.perf_counter()
            g = step(theta, order)
            theta = orn.sgd(theta, g, lr)
            t_total += time.perf_counter() - t0
            useful += int(data.lengths[order].sum())
            used.append(name)
            if t_total >= budget_s:
                break
        return useful, t_total, used

    pool = opool.Pool()
    try:
        # one untimed batch starts the workers and loads their imports
        pool.submit(m, data.params, data, sample[0][1][:pool.workers], need_tops=False).result()
        u_all, t_all, used_all = train(
            lambda th, order: pool.submit(m, th, data, order, need_tops=False).result()[1])
    finally:
        pool.close()

    def one_thread(theta, order):
        xs = [data.X[data.offsets[s]:data.offsets[s + 1]] for s in order]
        ys = [data.Y[data.offsets[s]:data.offsets[s + 1]] for s in order]
        return orn.forward_backward(m, theta, xs, ys)[1]

    with threadpool_limits(limits=1):
        u_one, t_one, used_one = train(one_thread, 1)
    cpu = cpu_model()
    return {"value": u_all / t_all, "unit": "timesteps/s", "cores": pool.workers,
            "kind": "oracle",
            "sample": (f"float64 oracle fwd+bwd+SGD (parameters carried from batch to batch) "
                       f"on the first batch of every bucket of epoch 0, then the longest "
                       f"batch, in that order until ~{budget_s:.0f} s: {', '.join(used_all)} "
                       f"({u_all} useful timesteps, {t_all:.1f} s); each batch's sequences "
                       f"split over {pool.workers} worker processes with one BLAS thread each, "
                       f"on {cpu}"),
            "one_thread": {"value": u_one / t_one, "cores": 1,
                           "sample": f"{', '.join(used_one)} ({u_one} useful timesteps, "
                                     f"{t_one:.1f} s, one thread)"}}


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3, help="timed steps (epochs)")
    ap.add_argument("--warmup", type=int, default=1, help="untimed epochs before them")
    ap.add_argument("--workload", default="bilstm3", choices=list(synth.WORKLOADS))
    ap.add_argument("--K", type=int, default=0, help="buckets (0 = largest of the workload)")
    ap.add_argument("--lr", type=float, default=0.1, help="SGD step size")
    ap.add_argument("--seed", type=int, default=0,
                    help="seed of the synthetic workload (lengths, data, parameters, shuffles)")
    ap.add_argument("--recurrence", default="resident", choices=("resident", "steps"),
                    help="resident kernels (default) or one launch per step "
                         "(the library's RNNBKT_RECURRENCE=steps)")
    ap.add_argument("--loss", default="frame", choices=("frame", "ctc"),
                    help="per-frame cross-entropy, or CTC over synthetic label strings "
                         "(one label per 8 frames)")
    ap.add_argument("--optimizer", default="sgd", choices=("sgd", "adadelta"),
                    help="parameter update of each step (adadelta: rho 0.95, eps 1e-6)")
    ap.add_argument("--ordering", default="ascending", choices=list(lib.ORDERINGS),
                    help="feeding order of the buckets / batches (the paper's: ascending)")
    ap.add_argument("--replicas", type=int, default=1,
                    help="R > 1: the headline is R replicas training at once on R streams, "
                         "each on its portion of the epoch, merged by eq. 3 (Sec. III.B)")
    ap.add_argument("--extra-replicas", type=int, default=0, metavar="R",
                    help="with --replicas 1, also measure R concurrent replicas over one epoch "
                         "and report them beside the headline (0 = skip)")
    ap.add_argument("--no-k1", action="store_true", help="skip the K=1 epoch")
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle baseline")
    ap.add_argument("--no-timer", action="store_true", help="skip the per-kernel pass")
    ap.add_argument("--calibrate", type=int, default=0, metavar="MIB",
                    help="first run rnnbkt_sgd_apply once over MIB MiB of parameters (reads "
                         "2x, writes 1x that many bytes): a streaming kernel of known size "
                         "for scaling hardware byte counters")
    args = ap.parse_args(argv)
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}, WORLD_SIZE {world}): "
              "the library runs on a single GPU; the paper's parallel scheme runs as concurrent "
              "replicas on that GPU (--replicas).", file=sys.stderr)
        return 2
    if args.steps < 1 or args.warmup < 0:
        print("--steps must be >= 1 and --warmup >= 0", file=sys.stderr)
        return 2
    if args.recurrence == "steps":
        os.environ["RNNBKT_RECURRENCE"] = "steps"  # read by the library at each call

    w = synth.WORKLOADS[args.workload]
    K = args.K or max(w.k_list)
    P = param_count(w)
    data = synth.make_workload(w, args.seed, param_count=P)
    # The oracle baseline runs first, before anything touches the GPU (its
    # worker processes are started fresh).
    cpu = None
    if not args.no_cpu and args.loss == "frame" and args.seed == 0:
        cpu = cpu_baseline(w, data, K, args.lr)

    import torch
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    lib.load()
    desc = lib.ModelDesc.of(w.cell, w.num_layers, w.input_dim, w.hidden, w.num_classes,
                            w.bidirectional, w.gemm_dtype)
    assert lib.param_count(desc) == P

    if args.calibrate:
        nf = args.calibrate * (1 << 20) // 4
        cp = torch.zeros(nf, dtype=torch.float32, device=dev)
        cg = torch.ones(nf, dtype=torch.float32, device=dev)
        lib.sgd_apply(cp, cg, 0.5)
        torch.cuda.synchronize()
        del cp, cg

    targets = (synth.ctc_targets(data.lengths, w.num_classes, args.seed) if args.loss == "ctc"
               else None)
    ep = Epoch(w, data, K, 0, torch, dev, targets, args.ordering, args.seed)
    ep1 = None if args.no_k1 else Epoch(w, data, 1, 0, torch, dev, targets, args.ordering,
                                        args.seed)
    eps = [e for e in (ep, ep1) if e is not None]
    rb, wb = lib.buffer_sizes(desc, max(e.max_T for e in eps), max(e.max_B for e in eps),
                              max(e.max_N for e in eps))
    reserve = torch.empty(rb, dtype=torch.uint8, device=dev)
    workspace = torch.empty(wb, dtype=torch.uint8, device=dev)
    params = torch.from_numpy(data.params).to(dev)
    grads = torch.zeros_like(params)
    loss = torch.zeros(1, dtype=torch.float32, device=dev)
    opt = None
    if args.optimizer == "adadelta":
        opt = (torch.zeros_like(params), torch.zeros_like(params))
    ctc_ws = None
    if targets is not None:
        nbytes = lib.ctc_workspace_bytes(max(e.max_T for e in eps), max(e.max_B for e in eps),
                                         max(e.max_U for e in eps))
        ctc_ws = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    state = (desc, params, grads, reserve, workspace, loss, args.lr, opt, ctc_ws)

    nb = len(ep.batches)
    ctc_bytes = None if ctc_ws is None else ctc_ws.numel()

    def replicated(R, e, warm, n_steps):
        lib.set_concurrency(R)
        try:
            rep = Replicated(R, desc, data, rb, wb, args.lr, args.optimizer, ctc_bytes, torch,
                             dev)
            return timed_replicated(e, rep, warm, n_steps, torch)
        finally:
            lib.set_concurrency(1)

    # The replicated figure is taken first: its streams then get hardware
    # queues of their own (the library's side stream, created by the first
    # sequential call, would otherwise share one with a replica).
    extra = None
    if args.replicas == 1 and args.extra_replicas > 1:
        extra = (args.extra_replicas,) + replicated(args.extra_replicas, ep, min(4, nb), nb)
    if args.replicas > 1:
        for _ in range(args.warmup):
            replicated(args.replicas, ep, 0, nb)
        secs_each = [replicated(args.replicas, ep, 0, nb)[1] for _ in range(args.steps)]
    else:
        secs_each = timed_epochs(ep, state, args.warmup, args.steps, torch)
    secs = sum(secs_each)
    value = args.steps * ep.U / secs
    rates = sorted(ep.U / t for t in secs_each)
    flops = flops_per_useful_step(w)
    peak = PEAK_TFLOPS[w.gemm_dtype]
    out = {
        "metric": METRIC, "value": value, "unit": "timesteps/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": secs * 1e3 / args.steps,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if w.gemm_dtype == synth.BF16 else "f32", "data": "synthetic",
        "config": {"workload": describe(w, K, args.seed),
                   "step": (f"one epoch: all {nb} batches of the epoch-0 schedule "
                            f"(buckets shortest first), each fwd + bwd + "
                            f"{args.optimizer} update; every timed step replays it"),
                   "loss": args.loss, "optimizer": args.optimizer,
                   "ordering": args.ordering, "recurrence": args.recurrence,
                   "batches_per_epoch": nb,
                   "useful_timesteps_per_epoch": ep.U,
                   "parallelism": "single GPU" if args.replicas == 1 else
                   f"{args.replicas} replicas on one GPU (concurrent streams, each a portion "
                   "of the epoch, merged by eq. 3 at its end)"},
        "epoch_rate_min": rates[0], "epoch_rate_max": rates[-1],
        "mfma_util_pct": 100.0 * flops * value / (peak * 1e12),
        "achieved_tflops": flops * value / 1e12,
        "pad_waste_pct": {"P_batch": 100.0 * (1 - ep.U / ep.p_batch),
                          "P_bucket": 100.0 * (1 - ep.U / ep.p_bucket),
                          "P_exec": 100.0 * (1 - ep.U / ep.p_exec)},
        "bucket_plan_ms": ep.plan_ms, "schedule_ms": ep.sched_ms,
        "bucket_upper": [int(u) for u in ep.upper],
    }
    if ep1 is not None:
        nb1 = len(ep1.batches)
        run_steps(ep1, state, 0, min(4, nb1), torch)  # warm the K=1 shapes
        if args.replicas > 1:
            s1 = replicated(args.replicas, ep1, 0, nb1)[1]
        else:
            (s1,) = timed_epochs(ep1, state, 0, 1, torch)
        out["k1"] = {"value": ep1.U / s1, "steps": 1, "batches": nb1, "ms_per_epoch": s1 * 1e3,
                     "pad_waste_pct_P_batch": 100.0 * (1 - ep1.U / ep1.p_batch),
                     "note": "one whole epoch at K=1 (random batches), timed as the headline"}
        out["speedup_vs_k1"] = value / (ep1.U / s1)

    if extra is not None:
        Rx, ux, sx = extra
        out["replicas"] = {
            "R": Rx, "value": ux / sx, "ms_per_epoch": sx * 1e3, "vs_sequential": ux / sx / value,
            "note": (f"the same batches dealt to {Rx} replicas training at once on {Rx} streams "
                     "(the paper's parallel scheme, Sec. III.B, on one GPU), merged by eq. 3 "
                     "at the end; a different optimisation trajectory from the sequential "
                     "headline")}
    if not args.no_timer and args.replicas == 1:
        torch.cuda.synchronize()
        lib.kernel_timer(True)
        run_steps(ep, state, 0, nb, torch)
        torch.cuda.synchronize()
        lib.kernel_timer(False)
        kinds = {k: lib.kernel_timer_read(k) for k in lib.KERNEL_KINDS}
        # Shares of the caller's stream; side-stream work overlaps the
        # recurrence and is reported beside them, as a fraction of the same total.
        crit = [k for k in kinds if k not in lib.OVERLAPPED_KINDS]
        total_ms = sum(kinds[k]["ms"] for k in crit)
        out["kernel_time_share"] = {k: round(kinds[k]["ms"] / total_ms, 4) for k in crit}
        out["overlapped_time_vs_stream"] = {k: round(kinds[k]["ms"] / total_ms, 4)
                                            for k in lib.OVERLAPPED_KINDS}
        dom = max(crit, key=lambda k: kinds[k]["ms"])
        d = kinds[dom]
        avg_s = d["ms"] / 1e3 / max(d["launches"], 1)
        if d["flops"] > 0:
            ach = d["flops"] / max(d["launches"], 1) / avg_s / 1e12
            roof = {"bound": "mfma", "achieved": ach, "peak": peak, "unit": "TFLOP/s",
                    "frac": ach / peak, "traffic": None}
        else:
            ach = d["bytes"] / max(d["launches"], 1) / avg_s / 1e9
            roof = {"bound": "hbm", "achieved": ach, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                    "frac": ach / PEAK_HBM_GBS, "traffic": None}
        roof["traffic"] = recorded_traffic(args.workload, K, dom)
        roof.update({"kernel": dom, "avg_launch_us": avg_s * 1e6, "launches": d["launches"]})
        out["roofline"] = roof
        out["kernels"] = {k: {"ms": v["ms"], "launches": v["launches"],
                              "avg_us": 1e3 * v["ms"] / max(v["launches"], 1)}
                          for k, v in kinds.items()}
        # Streaming kernels against the HBM roofline (algorithmic bytes).
        out["hbm_kernels"] = {
            k: {"GB/s": kinds[k]["bytes"] / (kinds[k]["ms"] / 1e3) / 1e9,
                "frac": kinds[k]["bytes"] / (kinds[k]["ms"] / 1e3) / 1e9 / PEAK_HBM_GBS,
                "bytes_per_launch": kinds[k]["bytes"] / max(kinds[k]["launches"], 1)}
            for k in ("xent", "sgd", "prepare") if k in kinds and kinds[k]["bytes"] > 0
            and kinds[k]["ms"] > 0}
        # Recurrence time per time step of the batches (the latency the
        # resident kernels are bound by; all layers of a launch together),
        # and per sequential step phase (layer or stack launch x step).
        t_sum = sum(int(L[0]) for L in ep.lens)
        out["recurrence_us_per_timestep"] = {
            "fwd": 1e3 * kinds["step_fwd"]["ms"] / t_sum,
            "bwd": 1e3 * kinds["step_bwd"]["ms"] / t_sum}
        if args.recurrence == "resident" and args.loss == "frame":
            out["latency_floor"] = latency_floor(w, ep, state, kinds, torch, dev)
    if cpu is not None:
        out["cpu_baseline"] = cpu
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
