"""Float64 connectionist temporal classification (CTC) loss and its gradient,
the training cost of the paper's experiments (Sec. IV.A): the network emits,
per frame, a distribution over the C output classes, class 0 being the blank;
a target is an unaligned label string l_1..l_U over classes 1..C-1; the loss
of a sequence is -ln p(l | x), p summing over every frame-level path that
collapses to l (merge repeated classes, then drop blanks).

Test infrastructure only (see oracle/__init__.py).

Written from the textbook definitions (Graves et al., 2006), in log space:
  extended target l' = (blank, l_1, blank, l_2, ..., l_U, blank), S = 2U + 1
  y_t(k)       softmax of the frame's logits z_t
  forward:     alpha_0(0) = y_0(blank), alpha_0(1) = y_0(l_1), 0 elsewhere;
               alpha_t(s) = (alpha_{t-1}(s) + alpha_{t-1}(s-1)
                             + [l'_s != blank and l'_s != l'_{s-2}] alpha_{t-1}(s-2))
                            * y_t(l'_s)
  backward:    beta_{T-1}(S-1) = y_{T-1}(blank), beta_{T-1}(S-2) = y_{T-1}(l_U);
               beta_t(s) = (beta_{t+1}(s) + beta_{t+1}(s+1)
                            + [l'_s != blank and l'_s != l'_{s+2}] beta_{t+1}(s+2))
                           * y_t(l'_s)
  p            = alpha_{T-1}(S-1) + alpha_{T-1}(S-2)
               (= sum_s alpha_t(s) beta_t(s) / y_t(l'_s) for every t)
  gradient     d(-ln p)/dz_t(k) = y_t(k) - (1 / p) sum_{s : l'_s = k} alpha_t(s) beta_t(s) / y_t(l'_s)
"""
from __future__ import annotations

import numpy as np

BLANK = 0


def _logsumexp(a, axis=None):
    m = np.max(a, axis=axis, keepdims=True)
    m = np.where(np.isfinite(m), m, 0.0)
    with np.errstate(divide="ignore"):  # all terms -inf: the sum is 0, its log -inf
        out = m + np.log(np.sum(np.exp(a - m), axis=axis, keepdims=True))
    return np.squeeze(out, axis=axis) if axis is not None else out.reshape(())


def extend(target):
    """l' = blank, l_1, blank, ..., l_U, blank."""
    target = np.asarray(target, np.int64)
    ext = np.full(2 * len(target) + 1, BLANK, np.int64)
    ext[1::2] = target
    return ext


def ctc_loss_grad(z, target):
    """-ln p(target | z) and its gradient with respect to the logits z [T, C]
    (float64).  target: labels in 1..C-1, length U >= 1.  An infeasible target
    (no path of length T) gives +inf and a zero gradient."""
    z = np.asarray(z, np.float64)
    T, C = z.shape
    lp = z - _logsumexp(z, axis=1)[:, None]          # ln y_t(k)
    ext = extend(target)
    S = len(ext)
    NEG = -np.inf
    # the skip transition s-2 -> s is allowed into a label differing from l'_{s-2}
    skip = np.zeros(S, bool)
    skip[2:] = (ext[2:] != BLANK) & (ext[2:] != ext[:-2])
    emit = lp[:, ext]                                 # ln y_t(l'_s)  [T, S]
    la = np.full((T, S), NEG)
    la[0, 0] = emit[0, 0]
    if S > 1:
        la[0, 1] = emit[0, 1]
    for t in range(1, T):
        prev = la[t - 1]
        stay = prev                                                  # s -> s
        step = np.concatenate(([NEG], prev[:-1]))                    # s-1 -> s
        jump = np.where(skip, np.concatenate(([NEG, NEG], prev[:-2])), NEG)  # s-2 -> s
        la[t] = np.logaddexp(np.logaddexp(stay, step), jump) + emit[t]
    # the transition s -> s+2 exists where the skip into s+2 does
    skip_from = np.concatenate((skip[2:], [False, False]))
    lb = np.full((T, S), NEG)
    lb[T - 1, S - 1] = emit[T - 1, S - 1]
    if S > 1:
        lb[T - 1, S - 2] = emit[T - 1, S - 2]
    for t in range(T - 2, -1, -1):
        nxt = lb[t + 1]
        stay = nxt                                                   # s <- s
        step = np.concatenate((nxt[1:], [NEG]))                      # s <- s+1
        jump = np.where(skip_from, np.concatenate((nxt[2:], [NEG, NEG])), NEG)  # s <- s+2
        lb[t] = np.logaddexp(np.logaddexp(stay, step), jump) + emit[t]
    ends = [la[T - 1, S - 1]] + ([la[T - 1, S - 2]] if S > 1 else [])
    lnp = _logsumexp(np.array(ends))
    if not np.isfinite(lnp):
        return np.inf, np.zeros_like(z)
    # occupancy of each extended state: alpha beta / y, normalised by p
    occ = np.exp(la + lb - emit - lnp)
    grad = np.exp(lp)
    for s in range(S):
        grad[:, ext[s]] -= occ[:, s]
    return float(-lnp), grad
