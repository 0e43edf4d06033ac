"""Reporting of waits that gave up, in the only form that keeps every kernel
well behaved: the host sets a poll budget of zero (RNNBKT_MAX_POLLS=0), so a
wait of a resident launch gives up at its first miss and reads on; every
launch still runs to its end.  rnnbkt_sync_check must report it once, and
launches after the report must be unaffected."""
import numpy as np
import pytest

from paper_1708_05604_amd import lib
from tests import harness as H

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lib.load()


@pytest.mark.parametrize("label,spec,lengths", [
    ("stack", H.Spec(0, 2, 0, 8, 64, 8), [60, 55, 40, 3]),
    ("bidirectional", H.Spec(0, 2, 1, 4, 32, 8), [50, 41, 7, 1]),
])
def test_timeout_reported_once_then_cleared(label, spec, lengths, monkeypatch):
    data = H.data_from_lengths(spec, lengths, seed=57, scale=0.3)
    order = H.batch_order(data, range(len(lengths)))
    lib.sync_check()  # nothing pending from earlier tests
    monkeypatch.setenv("RNNBKT_MAX_POLLS", "0")
    g = H.GpuBatch(spec, data.params, data, order)
    g.forward()
    g.backward()
    g.torch.cuda.synchronize()
    with pytest.raises(lib.RnnbktError) as e:
        lib.sync_check()
    assert e.value.code == lib.EHIP
    print(f"[case] {label}: {e.value}", flush=True)
    lib.sync_check()  # reported once: the count was cleared
    monkeypatch.delenv("RNNBKT_MAX_POLLS")
    # The next launches wait normally and match the oracle.
    H.assert_batch_close(spec, data.params, data, order, label=f"after timeout {label}")
    lib.sync_check()
