"""Pins of the float64 CTC oracle (oracle/ctc.py)."""
import itertools

import numpy as np
import pytest

from oracle import ctc


def _torch_ctc(z, target):
    """PyTorch's CPU CTC loss (float64) and its autograd gradient."""
    import torch
    zt = torch.tensor(z, dtype=torch.float64, requires_grad=True)
    lp = torch.log_softmax(zt, dim=1)[:, None, :]
    loss = torch.nn.functional.ctc_loss(
        lp, torch.tensor([list(target)], dtype=torch.long), torch.tensor([z.shape[0]]),
        torch.tensor([len(target)]), blank=0, reduction="sum", zero_infinity=False)
    loss.backward()
    return float(loss.detach()), zt.grad.numpy()


def _collapse(path):
    out, prev = [], None
    for k in path:
        if k != prev and k != ctc.BLANK:
            out.append(k)
        prev = k
    return tuple(out)


def _brute(z, target):
    """p by enumerating every frame-level path, and d(-ln p)/dz from the same sums."""
    T, C = z.shape
    y = np.exp(z - z.max(1, keepdims=True))
    y /= y.sum(1, keepdims=True)
    p = 0.0
    occ = np.zeros((T, C))  # sum of probabilities of matching paths with pi_t = k
    for path in itertools.product(range(C), repeat=T):
        if _collapse(path) != tuple(target):
            continue
        pr = np.prod([y[t, k] for t, k in enumerate(path)])
        p += pr
        for t, k in enumerate(path):
            occ[t, k] += pr
    return p, y - occ / p


@pytest.mark.parametrize("seed", range(12))
def test_matches_torch_ctc(seed):
    rng = np.random.default_rng(seed)
    C = int(rng.choice([3, 5, 20]))
    U = int(rng.integers(1, 8))
    target = rng.integers(1, C, U)
    if seed % 3 == 0 and U > 1:
        target[1] = target[0]  # a repeated label (needs a blank between)
    reps = int(np.sum(target[1:] == target[:-1]))
    T = int(rng.integers(U + reps, U + reps + 25))
    z = rng.standard_normal((T, C)) * 2.0
    loss, grad = ctc.ctc_loss_grad(z, target)
    tl, tg = _torch_ctc(z, target)
    assert abs(loss - tl) <= 1e-10 * abs(tl)
    np.testing.assert_allclose(grad, tg, rtol=1e-9, atol=1e-12)


@pytest.mark.parametrize("T,target", [(1, [1]), (3, [1]), (4, [1, 2]), (5, [2, 2]), (6, [1, 2, 1]),
                                      (6, [2, 2, 2]), (5, [1, 1])])
def test_matches_brute_force(T, target):
    rng = np.random.default_rng(T * 10 + len(target))
    z = rng.standard_normal((T, 3))
    loss, grad = ctc.ctc_loss_grad(z, target)
    p, g = _brute(z, target)
    assert abs(loss + np.log(p)) < 1e-12
    np.testing.assert_allclose(grad, g, atol=1e-12)


def test_single_path_when_target_fills_the_frames():
    """T = U and no repeated labels: the only path is the target itself."""
    rng = np.random.default_rng(3)
    target = np.array([3, 1, 4, 1, 5, 2])
    z = rng.standard_normal((6, 7))
    y = np.exp(z - z.max(1, keepdims=True))
    y /= y.sum(1, keepdims=True)
    loss, grad = ctc.ctc_loss_grad(z, target)
    assert abs(loss + np.sum(np.log(y[np.arange(6), target]))) < 1e-12
    onehot = np.zeros_like(y)
    onehot[np.arange(6), target] = 1.0
    np.testing.assert_allclose(grad, y - onehot, atol=1e-14)


def test_rows_sum_to_zero_and_shift_invariance():
    """Each frame's occupancies sum to one, so gradient rows sum to zero; a
    constant added to one frame's logits changes nothing."""
    rng = np.random.default_rng(5)
    target = rng.integers(1, 10, 12)
    z = rng.standard_normal((60, 10)) * 3.0
    loss, grad = ctc.ctc_loss_grad(z, target)
    np.testing.assert_allclose(grad.sum(1), 0.0, atol=1e-12)
    z2 = z.copy()
    z2[17] += 40.0
    loss2, grad2 = ctc.ctc_loss_grad(z2, target)
    assert abs(loss - loss2) < 1e-10
    np.testing.assert_allclose(grad, grad2, atol=1e-12)


def test_infeasible_target():
    """Equal adjacent labels need a blank between them, so three frames carry
    (1, 1) but not (1, 1, 1); fewer frames than labels carry nothing."""
    z = np.zeros((3, 4))
    assert ctc.ctc_loss_grad(z, [1, 1])[0] < np.inf
    loss, grad = ctc.ctc_loss_grad(z, [1, 1, 1])
    assert loss == np.inf and not grad.any()
    assert ctc.ctc_loss_grad(z, [1, 2, 3, 1])[0] == np.inf
