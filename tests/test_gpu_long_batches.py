"""GPU parity on the longest batches of the full-size workloads.

A batch costs its longest sequence (Sec. III.A, eq. 1): these are the
batches where the recurrences run longest (up to 4000 steps) and where bf16
operand rounding has the most steps to accumulate.  Each batch is the one
holding the longest sequence in epoch 0's schedule (ties: the most frames)
at the given bucket count; K = 1 is the paper's unbucketed baseline (random
batches).  The oracle runs in worker processes started at the beginning of
the session (tests/long_refs.py).  Bar: 1e-4 (fp32 GEMMs) or 2e-2 (bf16 GEMM
operands), normwise per tensor and per parameter block; element-wise
relative errors are logged beside it.
"""
import numpy as np
import pytest

from paper_1708_05604_amd import lib, synth
from tests import harness as H
from tests import long_refs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lib.load()


@pytest.mark.long_oracle
@pytest.mark.timeout(1500)
@pytest.mark.parametrize("name,K,T,B,N", long_refs.CASES,
                         ids=[long_refs.case_id(c[0], c[1]) for c in long_refs.CASES])
def test_longest_batch(name, K, T, B, N):
    w = synth.WORKLOADS[name]
    data, order, job = long_refs.get(long_refs.case_id(name, K))
    lens = data.lengths[order]
    assert (int(lens.max()), len(order), int(lens.sum())) == (T, B, N)
    # The library's planner and schedule pick the same batch.
    _, bof, keff, _ = lib.bucket_plan(data.lengths, K)
    batches = lib.epoch_schedule(data.lengths, bof, keff, synth.shuffle_keys(0, 0, w.n), w.batch)
    assert any(len(bt) == len(order) and np.array_equal(bt, order) for bt in batches)
    H.assert_long_batch_close(H.Spec.of(w), data.params, data, order, job,
                              label=f"{name} K={K} longest")
