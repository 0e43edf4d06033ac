"""Pins of the eq. 3 aggregation oracle: a hand-worked case, the weight-decay
closed form for identical replicas, numpy's mean at beta = 0 (a library
routine the oracle does not use), and invariances."""
import numpy as np
import pytest

from oracle import aggregate as oa


def test_hand_worked():
    # mean of [1, 2] and [3, 6] is [2, 4]; minus 0.5 * [10, -20]
    v = oa.aggregate([np.array([1.0, 2.0]), np.array([3.0, 6.0])], np.array([10.0, -20.0]),
                     beta=0.5)
    np.testing.assert_array_equal(v, [-3.0, 14.0])


def test_identical_replicas_decay():
    # every replica returned the previous values: V(t) = (1 - beta) V(t-1)
    rng = np.random.default_rng(0)
    prev = rng.standard_normal(100)
    for R in (1, 2, 6):
        v = oa.aggregate([prev.copy() for _ in range(R)], prev)
        np.testing.assert_allclose(v, (1.0 - oa.BETA) * prev, rtol=1e-15, atol=0)


@pytest.mark.parametrize("R", [1, 2, 3, 8])
def test_zero_beta_is_numpy_mean(R):
    rng = np.random.default_rng(R)
    reps = [rng.standard_normal(257) for _ in range(R)]
    v = oa.aggregate(reps, rng.standard_normal(257), beta=0.0)
    np.testing.assert_allclose(v, np.mean(np.stack(reps), axis=0), rtol=1e-15, atol=1e-16)


def test_invariances():
    rng = np.random.default_rng(5)
    reps = [rng.standard_normal(50) for _ in range(4)]
    prev = rng.standard_normal(50)
    a = oa.aggregate(reps, prev)
    b = oa.aggregate(reps[::-1], prev)
    np.testing.assert_allclose(a, b, rtol=1e-15, atol=1e-15)
    # linear in (replicas, prev) jointly
    c = oa.aggregate([2.0 * r for r in reps], 2.0 * prev)
    np.testing.assert_allclose(c, 2.0 * a, rtol=1e-14, atol=1e-15)
    with pytest.raises(ValueError):
        oa.aggregate([], prev)
