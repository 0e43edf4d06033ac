"""GPU parity of the CTC loss path (rnnbkt_lstm_fwd_ctc + rnnbkt_lstm_bwd)
against the float64 oracle (oracle/ctc.py through oracle/rnn.py)."""
import numpy as np
import pytest

from oracle import rnn as orn
from paper_1708_05604_amd import lib, synth
from tests import harness as H

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lib.load()


def _targets(rng, lengths, C, frames_per_label=3, repeats=False):
    out = []
    for L in lengths:
        U = max(1, int(L) // frames_per_label)
        t = rng.integers(1, C, U).astype(np.int32)
        if repeats and U >= 3:
            t[1] = t[0]
            t[2] = t[0]
        out.append(t)
    return out


CASES = [
    # (label, spec, lengths, frames per label, repeated labels)
    ("lstm-1l", H.Spec(0, 1, 0, 4, 32, 12), [30, 22, 22, 9, 3, 1], 3, False),
    ("lstm-1l-repeats", H.Spec(0, 1, 0, 4, 32, 8), [40, 31, 12, 7], 3, True),
    ("lstm-2l-uni", H.Spec(0, 2, 0, 8, 64, 20), [25, 25, 17, 4, 2], 2, True),
    ("lstm-2l-bi", H.Spec(0, 2, 1, 8, 32, 8), [19, 13, 7, 3, 1], 3, False),
    ("gru-2l", H.Spec(1, 2, 0, 8, 96, 20), [33, 20, 20, 6], 4, True),
    ("lstm-bf16", H.Spec(0, 2, 1, 8, 64, 16, synth.BF16), [24, 18, 11, 4], 3, False),
    ("wide-classes", H.Spec(0, 1, 0, 16, 32, 1024), [12, 9], 2, False),
]


@pytest.mark.parametrize("label,spec,lengths,fpl,rep", CASES, ids=[c[0] for c in CASES])
def test_ctc_shapes(label, spec, lengths, fpl, rep):
    rng = np.random.default_rng(len(label))
    data = H.data_from_lengths(spec, lengths, seed=len(label) + 1, scale=0.3)
    tg = _targets(rng, lengths, spec.num_classes, fpl, rep)
    order = H.batch_order(data, range(len(lengths)))
    H.assert_batch_close(spec, data.params, data, order, label="ctc " + label, targets=tg)


def test_ctc_target_fills_the_sequence():
    """U = L without repeats (a single path), next to U = 1."""
    spec = H.Spec(0, 1, 0, 4, 32, 8)
    lengths = [9, 6, 1]
    data = H.data_from_lengths(spec, lengths, seed=4, scale=0.3)
    tg = [np.array([1, 2, 3, 4, 5, 6, 7, 1, 2], np.int32), np.array([3], np.int32),
          np.array([5], np.int32)]
    order = H.batch_order(data, range(3))
    H.assert_batch_close(spec, data.params, data, order, label="ctc single-path", targets=tg)


@pytest.mark.parametrize("U", [40, 100, 250, 500, 1000])
def test_ctc_long_targets(U):
    """Every states-per-lane width of the sequential kernel (1 .. 32)."""
    spec = H.Spec(0, 1, 0, 4, 32, 24)
    L = 2 * U + 7
    lengths = [L, L - 5, U]
    rng = np.random.default_rng(U)
    data = H.data_from_lengths(spec, lengths, seed=U, scale=0.3)
    tg = [rng.integers(1, 24, U).astype(np.int32), rng.integers(1, 24, U - 3).astype(np.int32),
          rng.integers(1, 24, max(1, U // 2)).astype(np.int32)]
    order = H.batch_order(data, range(3))
    H.assert_batch_close(spec, data.params, data, order, label=f"ctc U={U}", targets=tg)


def test_ctc_infeasible_target():
    """A target no path can produce: infinite loss, zero contribution to the
    gradient (the other sequences' gradient as the oracle computes it)."""
    spec = H.Spec(0, 1, 0, 4, 32, 8)
    lengths = [10, 3, 3]
    data = H.data_from_lengths(spec, lengths, seed=9, scale=0.3)
    tg = [np.array([1, 2, 3], np.int32), np.array([2, 2, 2], np.int32),
          np.array([4, 4], np.int32)]
    order = H.batch_order(data, range(3))
    gb = H.GpuBatch(spec, data.params, data, order, targets=tg)
    loss_g, grad_g, _ = gb.run()
    loss_r, grad_r, _ = H.oracle_batch(spec, data.params, data, order, targets=tg)
    assert loss_g == np.inf and loss_r == np.inf
    assert np.all(np.isfinite(grad_g))
    errs = H.block_errors(spec, grad_g, grad_r)
    assert max(errs.values()) < 1e-4, errs


def test_ctc_deterministic():
    spec = H.Spec(0, 2, 0, 8, 64, 20)
    lengths = [60, 41, 41, 30, 9]
    rng = np.random.default_rng(2)
    data = H.data_from_lengths(spec, lengths, seed=2, scale=0.3)
    tg = _targets(rng, lengths, 20, 3, True)
    order = H.batch_order(data, range(5))
    a = H.GpuBatch(spec, data.params, data, order, targets=tg).run()
    b = H.GpuBatch(spec, data.params, data, order, targets=tg).run()
    assert a[0] == b[0]
    np.testing.assert_array_equal(a[1], b[1])


def test_ctc_lstm2_full_size_batch():
    """A full batch of the benchmark workload (2-layer LSTM, H=128, C=80,
    B=64) from its longest bucket, with the synthetic label strings."""
    w = synth.WORKLOADS["lstm2"]
    spec = H.Spec.of(w)
    data = synth.make_workload(w, 0, param_count=orn.param_count(spec.model()))
    tg = synth.ctc_targets(data.lengths, w.num_classes, 0)
    upper, bof, keff, _ = lib.bucket_plan(data.lengths, 8)
    batches = lib.epoch_schedule(data.lengths, bof, keff, synth.shuffle_keys(0, 0, w.n), w.batch)
    order = max(batches, key=lambda o: int(data.lengths[o[0]]))
    H.assert_batch_close(spec, data.params, data, order, label="ctc lstm2 longest batch",
                         targets=tg)
