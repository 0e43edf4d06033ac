"""Pins of the float64 ADADELTA oracle (oracle/optim.py)."""
import numpy as np
import pytest

from oracle import optim


def _steps(theta, grads, rho=optim.RHO, eps=optim.EPS, lr=1.0):
    eg2 = np.zeros_like(theta)
    edx2 = np.zeros_like(theta)
    x = theta
    for g in grads:
        x, eg2, edx2 = optim.adadelta(x, g, eg2, edx2, rho, eps, lr)
    return x, eg2, edx2


@pytest.mark.parametrize("rho,eps,lr", [(0.95, 1e-6, 1.0), (0.9, 1e-4, 0.5), (0.0, 1e-8, 2.0)])
def test_matches_torch_adadelta(rho, eps, lr):
    """An independent implementation of the same method: PyTorch's CPU
    Adadelta in float64 (no weight decay)."""
    import torch
    rng = np.random.default_rng(7)
    theta = rng.standard_normal(257)
    grads = [rng.standard_normal(257) * 10.0 ** rng.integers(-4, 3) for _ in range(25)]
    x, _, _ = _steps(theta, grads, rho, eps, lr)
    p = torch.tensor(theta, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.Adadelta([p], lr=lr, rho=rho, eps=eps)
    for g in grads:
        p.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
    np.testing.assert_allclose(x, p.detach().numpy(), rtol=1e-13, atol=1e-15)


def test_constant_gradient_fixed_point():
    """With a constant gradient g both accumulators tend to g^2 (the fixed
    point of E = rho E + (1 - rho) (E + eps) g^2 / (g^2 + eps) is E = g^2), so
    the step tends to exactly -g.  With g^2 = eps the approach is geometric
    with rate (1 + rho) / 2."""
    g = np.array([1e-3, -1e-3])
    eg2 = np.zeros(2)
    edx2 = np.zeros(2)
    x = np.zeros(2)
    for _ in range(3000):
        prev = x
        x, eg2, edx2 = optim.adadelta(x, g, eg2, edx2)
    np.testing.assert_allclose(x - prev, -g, rtol=1e-12)
    np.testing.assert_allclose(eg2, g * g, rtol=1e-12)
    np.testing.assert_allclose(edx2, g * g, rtol=1e-12)


def test_zero_gradient_only_decays():
    rng = np.random.default_rng(1)
    theta = rng.standard_normal(5)
    eg2 = rng.random(5)
    edx2 = rng.random(5)
    x, e1, e2 = optim.adadelta(theta, np.zeros(5), eg2, edx2)
    np.testing.assert_array_equal(x, theta)
    np.testing.assert_allclose(e1, optim.RHO * eg2, rtol=1e-15)
    np.testing.assert_allclose(e2, optim.RHO * edx2, rtol=1e-15)


def test_first_step_from_zero_state():
    """From zero accumulators the first step is -sqrt(eps / ((1 - rho) g^2 + eps)) g:
    about -sqrt(eps / (1 - rho)) sign(g) for large |g| (the method's slow start)."""
    g = np.array([1e-4, -0.5, 3.0, 1e3])
    x, eg2, edx2 = optim.adadelta(np.zeros(4), g, np.zeros(4), np.zeros(4))
    rho, eps = optim.RHO, optim.EPS
    np.testing.assert_allclose(x, -np.sqrt(eps / ((1 - rho) * g * g + eps)) * g, rtol=1e-14)
    np.testing.assert_allclose(eg2, (1 - rho) * g * g, rtol=1e-15)
    assert abs(x[-1] + np.sqrt(eps / (1 - rho))) < 1e-9
    assert np.all(np.sign(x) == -np.sign(g))
