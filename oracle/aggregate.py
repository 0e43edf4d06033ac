"""Float64 epoch-end aggregation of parallel replicas (paper Sec. III.B,
step 5, eq. 3).

Test infrastructure only (see oracle/__init__.py).

Each training process returns its parameters at the end of an epoch; with
the paper's choice alpha = 1 the aggregated parameters are the mean over the
R replicas minus a small decay proportional to the previous epoch's values:
    V(t) = V_alpha(t) - beta * V(t-1),   V_alpha(t) = (1/R) sum_r V_r(t),
beta = 1e-6 (the paper's value).  V(t-1) is the previous epoch's aggregate,
or the initial parameters for the first epoch.  Every replica starts the
next epoch from V(t).
"""
from __future__ import annotations

import numpy as np

BETA = 1e-6


def aggregate(replicas, prev, beta=BETA):
    """Eq. 3 in float64.  replicas: sequence of R parameter vectors (R >= 1);
    prev: V(t-1).  Returns V(t)."""
    R = len(replicas)
    if R < 1:
        raise ValueError("need at least one replica")
    total = np.zeros(np.shape(prev), np.float64)
    for v in replicas:
        total = total + np.asarray(v, np.float64)
    return total / R - beta * np.asarray(prev, np.float64)
