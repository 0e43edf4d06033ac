"""GPU parity: the library's HIP path against the float64 oracle on the same
seeded inputs (normwise relative error per tensor and per parameter block:
1e-4 for fp32 GEMMs, 2e-2 for bf16 GEMM operands)."""
import numpy as np
import pytest

from oracle import bucketing as ob
from oracle import rnn as orn
from oracle import schedule as osch
from paper_1708_05604_amd import lib, synth
from tests import harness as H

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lib.load()


def test_tiny_epoch_k2():
    """The whole tiny workload: planner, schedule, every batch fwd+bwd."""
    w = synth.WORKLOADS["tiny"]
    spec = H.Spec.of(w)
    P = orn.param_count(spec.model())
    data = synth.make_workload(w, 0, param_count=P)
    _, bof, keff, _ = lib.bucket_plan(data.lengths, 2)
    batches = lib.epoch_schedule(data.lengths, bof, keff, synth.shuffle_keys(0, 0, w.n), w.batch)
    for i, order in enumerate(batches):
        H.assert_batch_close(spec, data.params, data, order, label=f"tiny b{i}")


SHAPES = [
    # (label, spec, lengths)
    ("lstm-h64-b37-ragged", H.Spec(0, 1, 0, 4, 64, 12), [31, 30, 30, 29] + list(range(28, 0, -1))
     + [1, 1, 1, 1, 1]),
    ("lstm-2l-bi", H.Spec(0, 2, 1, 8, 32, 8), [9, 7, 7, 3, 1]),
    ("gru-2l-h96", H.Spec(1, 2, 0, 8, 96, 20), [17, 16, 12, 12, 12, 9, 5, 5, 4, 3, 2, 2, 1, 1, 1,
                                                1, 1, 1, 1, 1, 1]),
    ("gru-bi", H.Spec(1, 1, 1, 4, 32, 4), [6, 5, 2]),
    ("lstm-bf16-2l-bi", H.Spec(0, 2, 1, 8, 64, 16, synth.BF16), [20, 18, 11, 4, 4, 1]),
    ("gru-bf16", H.Spec(1, 1, 0, 8, 64, 16, synth.BF16), [20, 13, 2]),
    ("b1-t1", H.Spec(0, 1, 0, 4, 32, 4), [1]),
    ("equal-lengths", H.Spec(0, 1, 0, 4, 32, 8), [12] * 18),
    ("one-long", H.Spec(0, 2, 1, 4, 32, 8), [40, 1, 1, 1]),
    ("wide-classes", H.Spec(0, 1, 0, 16, 32, 1024), [5, 4]),
    # peephole LSTM (cell 2): uni/bi, a two-layer stack in one launch, bf16
    ("peep-h64-b37-ragged", H.Spec(2, 1, 0, 4, 64, 12), [31, 30, 30, 29]
     + list(range(28, 0, -1)) + [1, 1, 1, 1, 1]),
    ("peep-2l-bi", H.Spec(2, 2, 1, 8, 32, 8), [9, 7, 7, 3, 1]),
    ("peep-bf16-2l", H.Spec(2, 2, 0, 8, 64, 16, synth.BF16), [20, 18, 11, 4, 4, 1]),
    ("peep-one-long", H.Spec(2, 2, 0, 4, 32, 8), [40, 1, 1, 1]),
]


@pytest.mark.parametrize("label,spec,lengths", SHAPES, ids=[s[0] for s in SHAPES])
def test_shapes(label, spec, lengths):
    data = H.data_from_lengths(spec, lengths, seed=len(label), scale=0.3)
    order = H.batch_order(data, range(len(lengths)))
    H.assert_batch_close(spec, data.params, data, order, label=label)


STEP_SHAPES = [s for s in SHAPES if s[0] in ("lstm-h64-b37-ragged", "lstm-2l-bi", "gru-bi",
                                              "lstm-bf16-2l-bi", "gru-bf16", "one-long",
                                              "peep-h64-b37-ragged", "peep-2l-bi",
                                              "peep-bf16-2l")]


@pytest.mark.parametrize("label,spec,lengths", STEP_SHAPES, ids=[s[0] for s in STEP_SHAPES])
def test_shapes_per_step_kernels(label, spec, lengths, monkeypatch):
    """The one-launch-per-step recurrence kernels (the alternative to the
    persistent ones) on the same cases."""
    monkeypatch.setenv("RNNBKT_RECURRENCE", "steps")
    data = H.data_from_lengths(spec, lengths, seed=len(label), scale=0.3)
    order = H.batch_order(data, range(len(lengths)))
    H.assert_batch_close(spec, data.params, data, order, label="steps " + label)


def test_persistent_and_per_step_agree():
    """Both recurrence implementations give the same numbers (to rounding)."""
    import os
    spec = H.Spec(0, 2, 1, 8, 64, 12)
    data = H.data_from_lengths(spec, [33, 20, 20, 7, 7, 7, 2, 1, 1], seed=3, scale=0.3)
    order = H.batch_order(data, range(9))
    a = H.GpuBatch(spec, data.params, data, order).run()
    os.environ["RNNBKT_RECURRENCE"] = "steps"
    try:
        b = H.GpuBatch(spec, data.params, data, order).run()
    finally:
        del os.environ["RNNBKT_RECURRENCE"]
    assert abs(a[0] - b[0]) <= 1e-6 * abs(b[0])
    assert H.normwise_err(a[1], b[1]) < 1e-5
    assert H.normwise_err(a[2], b[2]) < 1e-5


def test_sgd_trajectory_tiny():
    """Three SGD steps on one batch: parameters follow the oracle's."""
    spec = H.Spec(0, 1, 0, 4, 32, 20)
    data = H.data_from_lengths(spec, [30, 22, 22, 9, 3], seed=5, scale=0.3)
    order = H.batch_order(data, range(5))
    lr = 0.5
    gb = H.GpuBatch(spec, data.params, data, order)
    theta = data.params.astype(np.float64)
    for step in range(3):
        gb.run()
        gb.sgd(lr)
        _, grad, _ = H.oracle_batch(spec, theta, data, order)
        theta = orn.sgd(theta, grad, lr)
        got = gb.params.cpu().numpy().astype(np.float64)
        err = H.normwise_err(got - data.params, theta - data.params)
        print(f"[case] sgd step {step} update err {err:.2e}", flush=True)
        assert err < 1e-4


@pytest.mark.parametrize("ordering", ["descending", "shuffled_batches"])
def test_epoch_sgd_under_feeding_order(ordering):
    """One SGD epoch over the tiny workload (K=2) fed in another order: the
    library's schedule equals the oracle's, and the parameters carried batch
    after batch follow the oracle's trajectory."""
    from oracle import schedule as osch
    w = synth.WORKLOADS["tiny"]
    spec = H.Spec.of(w)
    P = orn.param_count(spec.model())
    data = synth.make_workload(w, 0, param_count=P)
    _, bof, keff, _ = lib.bucket_plan(data.lengths, 2)
    keys, ok = synth.shuffle_keys(0, 3, w.n), synth.order_keys(0, 3, w.n)
    batches = lib.epoch_schedule(data.lengths, bof, keff, keys, w.batch, ordering, ok)
    ref = osch.epoch_batches(data.lengths, bof, keff, keys, w.batch, ordering, ok)
    assert [b.tolist() for b in batches] == [b.tolist() for b in ref]
    lr = 0.2
    p0 = data.params.astype(np.float64)
    cur = data.params.astype(np.float32)
    theta = p0.copy()
    for i, order in enumerate(batches):
        gb = H.GpuBatch(spec, cur, data, order)
        gb.run()
        gb.sgd(lr)
        cur = gb.params.cpu().numpy()
        _, grad, _ = H.oracle_batch(spec, theta, data, order)
        theta = orn.sgd(theta, grad, lr)
        err = H.normwise_err(cur.astype(np.float64) - p0, theta - p0)
        print(f"[case] {ordering} batch {i} B={len(order)} update err {err:.2e}", flush=True)
        assert err < 1e-4


def test_resume_at_epoch_boundary_is_exact(tmp_path):
    """Checkpoint / resume: the epoch's shuffle is derived from (seed, epoch)
    and every reduction runs in a fixed order, so two SGD epochs in a row equal
    one epoch, the flat parameter vector saved to a file and loaded back, and
    the second epoch -- bit for bit."""
    w = synth.WORKLOADS["tiny"]
    spec = H.Spec.of(w)
    data = synth.make_workload(w, 0, param_count=orn.param_count(spec.model()))
    _, bof, keff, _ = lib.bucket_plan(data.lengths, 2)
    lr = 0.2

    def epoch(params, e):
        keys = synth.shuffle_keys(0, e, w.n)
        cur = params
        for order in lib.epoch_schedule(data.lengths, bof, keff, keys, w.batch):
            gb = H.GpuBatch(spec, cur, data, order)
            gb.run()
            gb.sgd(lr)
            cur = gb.params.cpu().numpy()
        return cur

    p0 = data.params.astype(np.float32)
    straight = epoch(epoch(p0, 0), 1)
    ckpt = tmp_path / "params_epoch1.npy"
    np.save(ckpt, epoch(p0, 0))
    resumed = epoch(np.load(ckpt), 1)
    assert np.isfinite(straight).all()
    assert np.array_equal(straight, resumed)
    assert not np.array_equal(straight, p0)


def test_sgd_apply_exact():
    import torch
    rng = np.random.default_rng(0)
    for n in (1, 5, 1027, 4096):
        p = rng.standard_normal(n).astype(np.float32)
        g = rng.standard_normal(n).astype(np.float32)
        tp = torch.from_numpy(p).cuda()
        tg = torch.from_numpy(g).cuda()
        lib.sgd_apply(tp, tg, 0.25)
        torch.cuda.synchronize()
        ref = p.astype(np.float64) - 0.25 * g.astype(np.float64)
        np.testing.assert_allclose(tp.cpu().numpy(), ref, rtol=1e-6, atol=1e-7)


def test_adadelta_apply_matches_oracle():
    """Three consecutive ADADELTA steps on ragged sizes, gradients spanning
    eight decades, against the float64 oracle (state carried on both sides)."""
    import torch
    from oracle import optim
    rng = np.random.default_rng(11)
    for n in (1, 5, 1027, 4099):
        p = rng.standard_normal(n).astype(np.float32)
        tp = torch.from_numpy(p).cuda()
        ta = torch.zeros(n, dtype=torch.float32, device="cuda")
        tb = torch.zeros(n, dtype=torch.float32, device="cuda")
        x, e1, e2 = p.astype(np.float64), np.zeros(n), np.zeros(n)
        for step in range(3):
            g = (rng.standard_normal(n) * 10.0 ** rng.integers(-4, 4, n)).astype(np.float32)
            lib.adadelta_apply(tp, torch.from_numpy(g).cuda(), ta, tb)
            x, e1, e2 = optim.adadelta(x, g, e1, e2)
            torch.cuda.synchronize()
            for name, got, ref in (("params", tp, x), ("E[g^2]", ta, e1), ("E[dx^2]", tb, e2)):
                got = got.cpu().numpy().astype(np.float64)
                np.testing.assert_allclose(got, ref, rtol=1e-5, atol=1e-12 * np.max(np.abs(ref)),
                                           err_msg=f"n={n} step={step} {name}")


def test_adadelta_trajectory_tiny():
    """Three training steps (forward, backward, ADADELTA) on one batch: the
    parameters follow the oracle's trajectory."""
    import torch
    from oracle import optim
    spec = H.Spec(0, 1, 0, 4, 32, 20)
    data = H.data_from_lengths(spec, [30, 22, 22, 9, 3], seed=6, scale=0.3)
    order = H.batch_order(data, range(5))
    gb = H.GpuBatch(spec, data.params, data, order)
    ta = torch.zeros_like(gb.params)
    tb = torch.zeros_like(gb.params)
    theta = data.params.astype(np.float64)
    e1 = np.zeros_like(theta)
    e2 = np.zeros_like(theta)
    for step in range(3):
        gb.forward()
        gb.backward()
        lib.adadelta_apply(gb.params, gb.grads, ta, tb)
        torch.cuda.synchronize()
        lib.sync_check()
        _, grad, _ = H.oracle_batch(spec, theta, data, order)
        theta, e1, e2 = optim.adadelta(theta, grad, e1, e2)
        got = gb.params.cpu().numpy().astype(np.float64)
        err = H.normwise_err(got - data.params, theta - data.params)
        print(f"[case] adadelta step {step} update err {err:.2e}", flush=True)
        assert err < 1e-4


def test_nan_padding_and_determinism():
    """Pad frames filled with NaN change nothing, and two runs are bitwise equal."""
    spec = H.Spec(0, 2, 1, 8, 64, 12)
    data = H.data_from_lengths(spec, [25, 20, 20, 7, 7, 7, 2], seed=9, scale=0.3)
    order = H.batch_order(data, range(7))
    a = H.GpuBatch(spec, data.params, data, order).run()
    b = H.GpuBatch(spec, data.params, data, order, pad_fill=float("nan")).run()
    c = H.GpuBatch(spec, data.params, data, order).run()
    for u, v in ((a, b), (a, c)):
        assert u[0] == v[0]
        assert np.array_equal(u[1], v[1])
        assert np.array_equal(u[2], v[2])


@pytest.mark.parametrize("b_f", [0.0, 40.0])
def test_closed_form_long_sequence(b_f):
    """Zero weights: gates of 1/2 (or a forget gate of exactly 1 with a bias of
    40), so the cell follows a closed form over 4000 steps."""
    T = 4000
    spec = H.Spec(0, 1, 0, 4, 32, 4)
    m = spec.model()
    p = {k: np.zeros(s) for k, s in orn.param_layout(m)}
    bg = np.linspace(-0.002, 0.002, 32) if b_f else np.linspace(-2, 2, 32)
    p[("b", 0, 0)][64:96] = bg
    p[("b", 0, 0)][32:64] = b_f
    theta = orn.pack(m, p).astype(np.float32)
    data = H.data_from_lengths(spec, [T, T, 3], seed=1)
    order = H.batch_order(data, range(3))
    gb = H.GpuBatch(spec, theta, data, order)
    gb.forward()
    import torch
    torch.cuda.synchronize()
    top = gb.top.cpu().numpy().astype(np.float64)
    t = np.arange(T)[:, None]
    tb = np.tanh(bg.astype(np.float32).astype(np.float64))[None, :]
    c = (t + 1.0) * 0.5 * tb if b_f else tb * (1.0 - 2.0 ** (-(t + 1.0)))
    h = 0.5 * np.tanh(c)
    for b in range(2):
        err = H.normwise_err(top[:, b], h)
        print(f"[case] closed form b_f={b_f} err {err:.2e}", flush=True)
        # fp32 bar; the running sum adds 4000 rounded terms (observed ~2e-5)
        assert err < 1e-4


def _workload_batches(name, K, epoch=0):
    w = synth.WORKLOADS[name]
    spec = H.Spec.of(w)
    P = orn.param_count(spec.model())
    data = synth.make_workload(w, 0, param_count=P)
    _, bof, keff, _ = lib.bucket_plan(data.lengths, K)
    batches = lib.epoch_schedule(data.lengths, bof, keff, synth.shuffle_keys(0, epoch, w.n),
                                 w.batch)
    return spec, data, bof, batches


def _first_of_bucket(data, bof, batches, bucket):
    for bt in batches:
        if bof[bt[0]] == bucket:
            return bt
    raise AssertionError("bucket not found")


def test_lstm2_bench_config_sampled():
    """The benchmarked configuration (2-layer LSTM, H=128, B=64, K=8): the
    first batch of the shortest and of the longest bucket, full size."""
    spec, data, bof, batches = _workload_batches("lstm2", 8)
    for bucket in (0, 7):
        order = _first_of_bucket(data, bof, batches, bucket)
        H.assert_batch_close(spec, data.params, data, order, label=f"lstm2 bucket {bucket}")


@pytest.mark.parametrize("name,K", [("bilstm3", 16), ("longtail", 16), ("gru2", 8),
                                    ("lstm2p", 8)])
def test_workload_sampled_first_bucket(name, K):
    spec, data, bof, batches = _workload_batches(name, K)
    order = _first_of_bucket(data, bof, batches, 0)
    H.assert_batch_close(spec, data.params, data, order, label=f"{name} bucket 0")


def test_gru_wide_layer_five_slots_padded_grid():
    """GRU with H = 352: the backward's reduction over the 3H = 1056 gate
    gradients is 66 chunks of 16, 5 per wave of 16 (the wide-layer variant),
    and B = 40 is 3 row groups, so the backward grid is padded to whole
    clusters per XCD with workgroups that exit at once."""
    spec = H.Spec(1, 2, 0, 8, 352, 8)
    rng = np.random.default_rng(37)
    lengths = sorted(rng.integers(1, 24, 40).tolist(), reverse=True)
    data = H.data_from_lengths(spec, lengths, seed=37, scale=0.3)
    order = H.batch_order(data, range(40))
    H.assert_batch_close(spec, data.params, data, order, label="GRU H=352 B=40")


def test_gru_forward_twelve_units_per_workgroup():
    """fp32 GRU with H = 192 and B = 176 (11 row groups): 8 units per
    workgroup would need more workgroups than the GPU has CUs, so the
    forward takes 12 per workgroup on a grid padded to whole row-group
    clusters per XCD."""
    spec = H.Spec(1, 2, 0, 8, 192, 8)
    rng = np.random.default_rng(43)
    lengths = sorted(rng.integers(1, 21, 176).tolist(), reverse=True)
    data = H.data_from_lengths(spec, lengths, seed=43, scale=0.3)
    order = H.batch_order(data, range(176))
    H.assert_batch_close(spec, data.params, data, order, label="GRU H=192 B=176")


def test_bf16_lstm_forward_sixteen_units_per_workgroup():
    """bf16 LSTM with H = 256 and B = 80 (5 row groups): the two layers with
    8 units per workgroup would need more workgroups than the GPU has CUs,
    so the forward takes 16 per workgroup on a padded grid.  Weights at the
    workloads' scale (U(-0.1, 0.1)): at 0.3 a 256-wide recurrence amplifies
    the bf16 operand rounding past the bound with 8 units per workgroup too
    (identical results)."""
    spec = H.Spec(0, 2, 0, 8, 256, 8, synth.BF16)
    rng = np.random.default_rng(47)
    lengths = sorted(rng.integers(1, 15, 80).tolist(), reverse=True)
    data = H.data_from_lengths(spec, lengths, seed=47, scale=0.1)
    order = H.batch_order(data, range(80))
    H.assert_batch_close(spec, data.params, data, order, label="bf16 LSTM H=256 B=80")


@pytest.mark.parametrize("B,launches", [(48, 1), (112, 2)])
def test_bf16_lstm_stack_packed_gate_gradients(B, launches):
    """bf16 LSTM, two layers of H = 512 (longtail's layer), whose backward
    publishes its gate gradients as packed bf16 pairs.  B = 48: both layers
    fit one resident backward launch (16 waves of 4 slots, no scratch), the
    lower layer multiplying the upper layer's packed gradients inside it.
    B = 112: one launch per layer, the gradient between them from the dX
    GEMM reading the packed gradients."""
    spec = H.Spec(0, 2, 0, 16, 512, 16, synth.BF16)
    rng = np.random.default_rng(53 + B)
    lengths = sorted(rng.integers(1, 25, B).tolist(), reverse=True)
    data = H.data_from_lengths(spec, lengths, seed=53 + B, scale=0.1)
    order = H.batch_order(data, range(B))
    lib.kernel_timer(True)
    try:
        H.assert_batch_close(spec, data.params, data, order, label=f"bf16 LSTM H=512 B={B}")
        n = lib.kernel_timer_read("step_bwd")["launches"]
    finally:
        lib.kernel_timer(False)
    assert n == launches, (n, launches)


@pytest.mark.parametrize("din", [4, 12])
def test_bf16_narrow_input_weight_gradient(din):
    """bf16 bidirectional LSTM whose bottom layer has a handful of input
    features, not a multiple of 8: its dW_ih (din columns of one 128-wide
    tile) is reduced over more than 1000 frames in several split-K slices,
    the last one ragged."""
    spec = H.Spec(0, 2, 1, din, 64, 8, synth.BF16)
    rng = np.random.default_rng(61 + din)
    lengths = sorted(rng.integers(17, 61, 32).tolist(), reverse=True)
    assert sum(lengths) > 1000 and sum(lengths) % 32 != 0
    data = H.data_from_lengths(spec, lengths, seed=61 + din, scale=0.1)
    order = H.batch_order(data, range(32))
    H.assert_batch_close(spec, data.params, data, order, label=f"bf16 BiLSTM din={din}")


def test_sequence_longer_than_resident_limit():
    """T_max above the 6144 steps whose batch tables the resident kernels keep
    in LDS: the recurrences fall back to one launch per step."""
    spec = H.Spec(0, 2, 0, 4, 32, 8)
    data = H.data_from_lengths(spec, [6200, 6150, 17, 1], seed=21, scale=0.3)
    order = H.batch_order(data, range(4))
    H.assert_batch_close(spec, data.params, data, order, label="T=6200 per-step fallback")


def test_wide_batch_many_row_groups():
    """B = 256 (16 row groups of 16 rows) with ragged lengths down to 1."""
    spec = H.Spec(0, 2, 0, 8, 64, 16)
    rng = np.random.default_rng(31)
    lengths = sorted(rng.integers(1, 41, 256).tolist(), reverse=True)
    data = H.data_from_lengths(spec, lengths, seed=31, scale=0.3)
    order = H.batch_order(data, range(256))
    H.assert_batch_close(spec, data.params, data, order, label="B=256")


def test_batch_beyond_single_launch_tables():
    """B = 300, more sequences than the one-launch batch preparation takes:
    tables and packing by the separate kernels."""
    spec = H.Spec(0, 2, 0, 4, 32, 8)
    rng = np.random.default_rng(33)
    lengths = sorted(rng.integers(1, 25, 300).tolist(), reverse=True)
    data = H.data_from_lengths(spec, lengths, seed=33, scale=0.3)
    order = H.batch_order(data, range(300))
    H.assert_batch_close(spec, data.params, data, order, label="B=300")


@pytest.mark.parametrize("label,spec,lengths", [
    ("stream-1l", H.Spec(0, 1, 0, 4, 64, 12), [31, 30, 30, 29] + list(range(28, 0, -1))),
    ("stream-2l", H.Spec(0, 2, 0, 8, 32, 8), [70, 64, 40, 33, 17, 17, 3, 1]),
    ("stream-peep-2l", H.Spec(2, 2, 0, 4, 32, 8), [50, 49, 20, 1]),
])
def test_streamed_weight_gradients(label, spec, lengths, monkeypatch):
    """Weight gradients computed beside the backward recurrence (fp32 LSTM
    stacks) match the oracle and the products computed after it (to
    rounding: the frames are summed in another order)."""
    data = H.data_from_lengths(spec, lengths, seed=41, scale=0.3)
    order = H.batch_order(data, range(len(lengths)))
    H.assert_batch_close(spec, data.params, data, order, label=label)
    a = H.GpuBatch(spec, data.params, data, order).run()
    monkeypatch.setenv("RNNBKT_WGRAD", "after")
    b = H.GpuBatch(spec, data.params, data, order).run()
    assert a[0] == b[0]
    assert H.normwise_err(a[1], b[1]) < 1e-6



@pytest.mark.parametrize("label,spec,lengths,env", [
    ("lstm-streamed", H.Spec(0, 2, 0, 8, 32, 8), [40, 33, 17, 2], {}),
    ("lstm-output-after", H.Spec(0, 2, 0, 8, 32, 8), [40, 33, 17, 2], {"RNNBKT_OUTPUT": "after"}),
    ("gru-bf16", H.Spec(1, 2, 0, 8, 32, 8, synth.BF16), [40, 33, 17, 2], {}),
    ("bilstm", H.Spec(0, 2, 1, 4, 32, 8), [30, 29, 3, 1], {}),
])
def test_backward_repeated_without_forward(label, spec, lengths, env, monkeypatch):
    """The forward leaves the backward's exchange buffers holding the
    sentinel; a second backward of the same batch (buffers now used) sets it
    itself, and both give the same gradients bit for bit."""
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    data = H.data_from_lengths(spec, lengths, seed=45, scale=0.3)
    order = H.batch_order(data, range(len(lengths)))
    g = H.GpuBatch(spec, data.params, data, order)
    g.forward()
    g.backward()
    g.torch.cuda.synchronize()
    first = g.grads.cpu().numpy().copy()
    g.grads.fill_(float("nan"))
    g.backward()
    g.torch.cuda.synchronize()
    lib.sync_check()
    second = g.grads.cpu().numpy()
    assert np.isfinite(first).all()
    assert np.array_equal(first, second), label


@pytest.mark.gpu
@pytest.mark.parametrize("label,spec,lengths", [
    ("out-1l-c12", H.Spec(0, 1, 0, 4, 64, 12), [31, 30, 30, 29] + list(range(28, 0, -1))),
    ("out-2l-tiny", H.Spec(0, 2, 0, 8, 32, 8), [9, 5, 3, 1]),
    ("out-2l-many-blocks", H.Spec(0, 2, 0, 8, 64, 20),
     [int(v) for v in np.linspace(140, 3, 48)]),
    ("out-peep-2l", H.Spec(2, 2, 0, 4, 32, 8), [50, 49, 20, 1]),
    ("out-bi-2l", H.Spec(0, 2, 1, 4, 32, 16), [37, 36, 18, 2]),
    ("out-gru-2l", H.Spec(1, 2, 0, 4, 32, 8), [44, 30, 29, 5]),
])
def test_streamed_output_layer(label, spec, lengths, monkeypatch):
    """The output layer and loss computed beside the forward recurrence
    (output-layer workgroups of the forward launch, blocks of 32 frames, more blocks than
    workgroups) match the oracle and the separate kernels run after it (to
    rounding: logits and loss are summed in another order)."""
    data = H.data_from_lengths(spec, lengths, seed=43, scale=0.3)
    order = H.batch_order(data, range(len(lengths)))
    H.assert_batch_close(spec, data.params, data, order, label=label)
    a = H.GpuBatch(spec, data.params, data, order).run()
    monkeypatch.setenv("RNNBKT_OUTPUT", "after")
    b = H.GpuBatch(spec, data.params, data, order).run()
    assert abs(a[0] - b[0]) <= 1e-6 * abs(b[0])
    assert H.normwise_err(a[1], b[1]) < 1e-5
