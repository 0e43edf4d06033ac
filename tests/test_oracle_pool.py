"""The split oracle (worker processes, N-weighted parts) equals the oracle run
on the whole batch in one process."""
import numpy as np

from oracle import rnn as orn
from paper_1708_05604_amd import synth
from tests import harness as H
from oracle import pool as opool


def test_pool_equals_single_process():
    spec = H.Spec(synth.LSTM, 2, 1, 4, 8, 5)
    lengths = [9, 7, 7, 5, 3, 2, 1]
    data = H.data_from_lengths(spec, lengths, seed=11, scale=0.3)
    order = H.batch_order(data, range(len(lengths)))
    loss_r, grad_r, top_r = H.oracle_batch(spec, data.params, data, order)
    pool = opool.Pool(workers=3)
    try:
        job = pool.submit(spec.model(), data.params, data, order, label="pool")
        assert len(job.groups) == 3
        loss_p, grad_p, tops_p = job.result()
    finally:
        pool.close()
    assert abs(loss_p - loss_r) <= 1e-13 * abs(loss_r)
    assert np.max(np.abs(grad_p - grad_r)) <= 1e-13 * np.max(np.abs(grad_r))
    for b, L in enumerate(data.lengths[order]):
        assert np.allclose(tops_p[b], top_r[:L, b], rtol=0, atol=1e-6)
