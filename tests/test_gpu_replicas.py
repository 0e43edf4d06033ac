"""Parallel replicas on one GPU (Sec. III.B): the eq. 3 aggregation kernel
against the float64 oracle, replicas trained on concurrent streams against
the same work run one after another, and a whole replicated epoch against
the oracle's replica trajectories and aggregation."""
import numpy as np
import pytest

from oracle import aggregate as oa
from oracle import rnn as orn
from paper_1708_05604_amd import lib, synth
from tests import harness as H

pytestmark = pytest.mark.gpu


def _within_one_ulp(got, ref):
    ref32 = ref.astype(np.float32)
    ulp = np.spacing(np.abs(ref32)).astype(np.float64)
    return np.abs(got.astype(np.float64) - ref) <= ulp


@pytest.mark.parametrize("R,n", [(1, 1), (2, 5), (3, 1027), (7, 300001), (16, 4096)])
def test_epoch_aggregate_matches_oracle(R, n):
    import torch
    rng = np.random.default_rng(R * 1000 + n)
    stride = (n + 3) // 4 * 4 + 8
    reps = rng.standard_normal((R, stride)).astype(np.float32)
    prev = rng.standard_normal(n).astype(np.float32) * 10
    beta = 1e-6 if R != 2 else 0.25
    print(f"[case] aggregate R={R} n={n} stride={stride} beta={beta}", flush=True)
    tr = torch.from_numpy(reps).cuda()
    tp = torch.from_numpy(prev).cuda()
    lib.epoch_aggregate(tr, tp, beta, n=n)
    torch.cuda.synchronize()
    ref = oa.aggregate([reps[r, :n] for r in range(R)], prev, beta)
    got_r = tr.cpu().numpy()
    got_p = tp.cpu().numpy()
    assert np.all(_within_one_ulp(got_p, ref))
    for r in range(R):
        assert np.all(_within_one_ulp(got_r[r, :n], ref))
        assert np.array_equal(got_r[r, n:], reps[r, n:])  # padding untouched


def _stage(data, batches):
    """Device copies of the batches' padded inputs (staged before any
    training call, so host copies never wait on a busy stream)."""
    import torch
    out = []
    for order in batches:
        x, y, lens = synth.padded_batch(data, order)
        out.append((torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda(), lens))
    torch.cuda.synchronize()
    return out


def _train(desc, bufs, staged, lr, stream):
    """SGD over the staged batches on one replica's buffers, on `stream`."""
    p, g, res, ws, loss = bufs
    for xd, yd, lens in staged:
        lib.lstm_fwd(desc, p, xd, yd, lens, res, ws, loss, stream=stream)
        lib.lstm_bwd(desc, p, lens, res, ws, g, stream=stream)
        lib.sgd_apply(p, g, lr, stream=stream)


def _buffers(spec, data, batches, count=1):
    import torch
    desc = spec.desc()
    T = max(int(data.lengths[b].max()) for b in batches)
    B = max(len(b) for b in batches)
    N = max(int(data.lengths[b].sum()) for b in batches)
    rb, wb = lib.buffer_sizes(desc, T, B, N)
    out = []
    for _ in range(count):
        out.append((torch.from_numpy(data.params.copy()).cuda(),
                    torch.zeros(len(data.params), dtype=torch.float32, device="cuda"),
                    torch.empty(rb, dtype=torch.uint8, device="cuda"),
                    torch.empty(wb, dtype=torch.uint8, device="cuda"),
                    torch.zeros(1, dtype=torch.float32, device="cuda")))
    return desc, out


@pytest.mark.parametrize("name,K,nb", [("tiny", 2, 4), ("lstm2", 8, 6)])
def test_concurrent_streams_match_sequential(name, K, nb):
    """Two replicas trained at once on two streams give bit-identical
    parameters to the same two trainings run one after the other."""
    import torch
    w = synth.WORKLOADS[name]
    spec = H.Spec.of(w)
    data = synth.make_workload(w, 0, param_count=orn.param_count(spec.model()))
    _, bof, keff, _ = lib.bucket_plan(data.lengths, K)
    batches = lib.epoch_schedule(data.lengths, bof, keff, synth.shuffle_keys(0, 0, w.n), w.batch)
    # one short and one long bucket's batches, so the two streams overlap
    # kernels of different sizes
    parts = [batches[:nb], batches[-nb:]]
    print(f"[case] {name} K={K} two streams x {nb} batches", flush=True)
    staged = [_stage(data, parts[r]) for r in range(2)]
    desc, seq = _buffers(spec, data, parts[0] + parts[1], 2)
    s0 = torch.cuda.current_stream()
    # Both runs with two streams declared, so both take the same kernels
    # (with one stream the backward would also overlap work of its own).
    lib.set_concurrency(2)
    try:
        for r in range(2):
            _train(desc, seq[r], staged[r], 0.1, s0)
        torch.cuda.synchronize()
        lib.sync_check()
    finally:
        lib.set_concurrency(1)
    _, con = _buffers(spec, data, parts[0] + parts[1], 2)
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    lib.set_concurrency(2)
    try:
        torch.cuda.synchronize()
        for k in range(nb):  # interleave the enqueues batch by batch
            for r in range(2):
                _train(desc, con[r], [staged[r][k]], 0.1, streams[r])
        torch.cuda.synchronize()
        lib.sync_check()
    finally:
        lib.set_concurrency(1)
    for r in range(2):
        assert torch.equal(seq[r][0], con[r][0]), f"replica {r} differs"


def test_replicated_epoch_matches_oracle():
    """The tiny workload's epoch split between two replicas (batches dealt in
    turn), each trained with SGD on its own stream, then merged by eq. 3:
    the merged parameters follow the oracle's."""
    import torch
    w = synth.WORKLOADS["tiny"]
    spec = H.Spec.of(w)
    data = synth.make_workload(w, 0, param_count=orn.param_count(spec.model()))
    _, bof, keff, _ = lib.bucket_plan(data.lengths, 2)
    batches = lib.epoch_schedule(data.lengths, bof, keff, synth.shuffle_keys(0, 0, w.n), w.batch)
    R, lr = 2, 0.2
    parts = [batches[r::R] for r in range(R)]
    print(f"[case] tiny replicated epoch R={R} batches {[len(p) for p in parts]}", flush=True)
    desc = spec.desc()
    P = len(data.params)
    stride = (P + 3) // 4 * 4
    reps = torch.zeros((R, stride), dtype=torch.float32, device="cuda")
    for r in range(R):
        reps[r, :P] = torch.from_numpy(data.params).cuda()
    prev = torch.from_numpy(data.params.copy()).cuda()
    grads = [torch.zeros(P, dtype=torch.float32, device="cuda") for _ in range(R)]
    rb, wb = lib.buffer_sizes(desc, int(data.lengths.max()), w.batch,
                              max(int(data.lengths[b].sum()) for b in batches))
    streams = [torch.cuda.Stream() for _ in range(R)]
    staged = [_stage(data, parts[r]) for r in range(R)]
    lib.set_concurrency(R)
    try:
        torch.cuda.synchronize()
        # every replica's buffers stay referenced until the streams are done
        bufs = [(reps[r, :P], grads[r], torch.empty(rb, dtype=torch.uint8, device="cuda"),
                 torch.empty(wb, dtype=torch.uint8, device="cuda"),
                 torch.zeros(1, dtype=torch.float32, device="cuda")) for r in range(R)]
        torch.cuda.synchronize()
        for r in range(R):
            _train(desc, bufs[r], staged[r], lr, streams[r])
        torch.cuda.synchronize()
        lib.epoch_aggregate(reps, prev, n=P)
        torch.cuda.synchronize()
        lib.sync_check()
    finally:
        lib.set_concurrency(1)
    theta0 = data.params.astype(np.float64)
    finals = []
    for r in range(R):
        theta = theta0.copy()
        for order in parts[r]:
            _, g, _ = H.oracle_batch(spec, theta, data, order)
            theta = orn.sgd(theta, g, lr)
        finals.append(theta)
    ref = oa.aggregate(finals, theta0)
    got = prev.cpu().numpy().astype(np.float64)
    err = H.normwise_err(got - theta0, ref - theta0)
    print(f"[case] replicated epoch update err {err:.2e}", flush=True)
    assert err < 1e-4
    for r in range(R):
        assert torch.equal(reps[r, :P], prev)
