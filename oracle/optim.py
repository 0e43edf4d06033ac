"""Float64 ADADELTA, the parameter update rule the paper's training processes
use (Sec. III.B, step 4, its ref. [21]: Zeiler, 2012).

Test infrastructure only (see oracle/__init__.py).

The paper names the method without its constants; Zeiler's defaults are
taken: decay rho = 0.95, conditioning constant eps = 1e-6, and a unit step
multiplier lr (the method itself has none; lr = 1 is the method as
published).  Both accumulators start at zero.  One update, in the order of
the method's algorithm:
    accumulate the squared gradient:  E[g^2] <- rho E[g^2] + (1 - rho) g^2
    compute the update:               dx = -(RMS[dx] / RMS[g]) g,
                                      RMS[y] = sqrt(E[y^2] + eps), with the
                                      E[dx^2] of the previous step
    accumulate the squared update:    E[dx^2] <- rho E[dx^2] + (1 - rho) dx^2
    apply the update:                 x <- x + lr dx
"""
from __future__ import annotations

import numpy as np

RHO = 0.95
EPS = 1e-6


def adadelta(theta, grad, acc_g2, acc_dx2, rho=RHO, eps=EPS, lr=1.0):
    """One ADADELTA step; returns (theta, acc_g2, acc_dx2), all float64 copies."""
    x = np.asarray(theta, np.float64).copy()
    g = np.asarray(grad, np.float64)
    eg2 = np.asarray(acc_g2, np.float64).copy()
    edx2 = np.asarray(acc_dx2, np.float64).copy()
    eg2 = rho * eg2 + (1.0 - rho) * g * g
    dx = -(np.sqrt(edx2 + eps) / np.sqrt(eg2 + eps)) * g
    edx2 = rho * edx2 + (1.0 - rho) * dx * dx
    x = x + lr * dx
    return x, eg2, edx2
