"""Float64 recurrent model, per-frame loss, backpropagation through time, SGD.

Test infrastructure only (see oracle/__init__.py).

The paper trains an LSTM (its ref. [1]) and names the GRU (ref. [2]) as the
lighter alternative (Sec. I); it prints no cell equations, so the standard
forms are used:

LSTM, gates in the order i, f, g, o, no peepholes, one bias per gate,
zero initial state:
    a_t = W_ih x_t + W_hh h_{t-1} + b
    i = sig(a_i), f = sig(a_f), g = tanh(a_g), o = sig(a_o)
    c_t = f * c_{t-1} + i * g,   h_t = o * tanh(c_t)
LSTM with peepholes (the paper trains its LSTM with Lasagne, Sec. IV.A,
whose LSTM layer has them by default): diagonal weights p_i, p_f, p_o let the
input and forget gates see the previous cell state and the output gate the
new one,
    i = sig(a_i + p_i * c_{t-1}), f = sig(a_f + p_f * c_{t-1}), g = tanh(a_g)
    c_t = f * c_{t-1} + i * g,   o = sig(a_o + p_o * c_t),   h_t = o * tanh(c_t)
GRU, gates r, z, n, the reset gate scaling the whole recurrent term of n:
    r = sig(W_ir x + b_ir + W_hr h + b_hr)
    z = sig(W_iz x + b_iz + W_hz h + b_hz)
    n = tanh(W_in x + b_in + r * (W_hn h + b_hn))
    h' = (1 - z) * n + z * h
A reverse direction runs over each sequence's own length, from its last frame
to its first; a bidirectional layer emits [h_fwd ; h_bwd] per frame and the
next layer (and the output layer) reads that concatenation.

Output: z_t = W_out h_t + b_out over the top layer, log-softmax, and the loss
is the mean over all valid frames of the batch of -log p_t[y_t] (the paper's
CTC loss is replaced by per-frame cross-entropy with one label per frame).
Pad frames do not exist here: every sequence is processed at its own length.

Flat parameter layout (float32 on the wire, float64 inside), row-major:
  for each layer, for each direction (forward first):
    W_ih [G*H, D_in], W_hh [G*H, H], then
    LSTM: b [4H]          GRU: b_ih [3H], b_hh [3H]
    LSTM with peepholes: b [4H], then p [3H] = (p_i, p_f, p_o)
  then W_out [C, H_top], b_out [C]
with G = 4 (LSTM) or 3 (GRU), D_in = input dim for layer 0 and
H * (2 if bidirectional else 1) above, H_top = the same width for the top.
"""
from __future__ import annotations

import dataclasses

import numpy as np

LSTM = 0
GRU = 1
LSTM_PEEPHOLE = 2


@dataclasses.dataclass(frozen=True)
class Model:
    cell: int
    num_layers: int
    bidirectional: int
    input_dim: int
    hidden: int
    num_classes: int

    @property
    def gates(self) -> int:
        return 3 if self.cell == GRU else 4

    @property
    def is_lstm(self) -> bool:
        return self.cell in (LSTM, LSTM_PEEPHOLE)

    @property
    def dirs(self) -> int:
        return 2 if self.bidirectional else 1

    def layer_input(self, layer: int) -> int:
        return self.input_dim if layer == 0 else self.hidden * self.dirs


def param_layout(m: Model):
    """List of (name, shape) in flat order; name = (kind, layer, direction)."""
    G, H = m.gates, m.hidden
    out = []
    for l in range(m.num_layers):
        for d in range(m.dirs):
            out.append((("W_ih", l, d), (G * H, m.layer_input(l))))
            out.append((("W_hh", l, d), (G * H, H)))
            if m.is_lstm:
                out.append((("b", l, d), (G * H,)))
                if m.cell == LSTM_PEEPHOLE:
                    out.append((("p", l, d), (3 * H,)))
            else:
                out.append((("b_ih", l, d), (G * H,)))
                out.append((("b_hh", l, d), (G * H,)))
    out.append((("W_out", 0, 0), (m.num_classes, H * m.dirs)))
    out.append((("b_out", 0, 0), (m.num_classes,)))
    return out


def param_count(m: Model) -> int:
    return int(sum(int(np.prod(s)) for _, s in param_layout(m)))


def unpack(m: Model, theta) -> dict:
    """Flat vector -> dict of float64 arrays (copies)."""
    theta = np.asarray(theta)
    p, pos = {}, 0
    for name, shape in param_layout(m):
        size = int(np.prod(shape))
        p[name] = theta[pos:pos + size].astype(np.float64).reshape(shape)
        pos += size
    assert pos == theta.size, (pos, theta.size)
    return p


def pack(m: Model, p: dict) -> np.ndarray:
    return np.concatenate([np.asarray(p[name], np.float64).reshape(-1)
                           for name, _ in param_layout(m)])


def _sig(x):
    return 1.0 / (1.0 + np.exp(-x))


def _time_order(L: int, d: int):
    return range(L) if d == 0 else range(L - 1, -1, -1)


def lstm_dir_forward(W_ih, W_hh, b, X, d, peep=None):
    """One direction of one LSTM layer over one sequence X [L, D_in];
    `peep` = [p_i ; p_f ; p_o] (3H) for the peephole cell, else None.
    Returns (Hseq [L, H], cache)."""
    L = X.shape[0]
    H = W_hh.shape[1]
    p_i, p_f, p_o = (np.zeros(H),) * 3 if peep is None else np.reshape(peep, (3, H))
    ax = X @ W_ih.T + b                           # input part of a_t, all t
    Hs = np.zeros((L, H))
    cache = {"i": np.zeros((L, H)), "f": np.zeros((L, H)), "g": np.zeros((L, H)),
             "o": np.zeros((L, H)), "c": np.zeros((L, H)), "c_prev": np.zeros((L, H)),
             "h_prev": np.zeros((L, H))}
    h = np.zeros(H)
    c = np.zeros(H)
    for t in _time_order(L, d):
        a = ax[t] + W_hh @ h
        i = _sig(a[0:H] + p_i * c)
        f = _sig(a[H:2 * H] + p_f * c)
        g = np.tanh(a[2 * H:3 * H])
        cache["h_prev"][t] = h
        cache["c_prev"][t] = c
        c = f * c + i * g
        o = _sig(a[3 * H:4 * H] + p_o * c)
        h = o * np.tanh(c)
        Hs[t] = h
        for k, v in (("i", i), ("f", f), ("g", g), ("o", o), ("c", c)):
            cache[k][t] = v
    return Hs, cache


def lstm_dir_backward(W_ih, W_hh, X, cache, dH, d, peep=None):
    """Reverse-mode pass of ``lstm_dir_forward`` given dLoss/dh_t = dH [L, H].
    Returns (dW_ih, dW_hh, db, dX, dpeep); dpeep (3H) is zero without
    peepholes."""
    L = X.shape[0]
    H = W_hh.shape[1]
    p_i, p_f, p_o = (np.zeros(H),) * 3 if peep is None else np.reshape(peep, (3, H))
    dA = np.zeros((L, 4 * H))
    dh_rec = np.zeros(H)      # gradient reaching h_t through the next step's W_hh
    dc_rec = np.zeros(H)      # gradient reaching c_t through the next step's gates
    for t in reversed(list(_time_order(L, d))):
        i, f, g, o = cache["i"][t], cache["f"][t], cache["g"][t], cache["o"][t]
        c, c_prev, h_prev = cache["c"][t], cache["c_prev"][t], cache["h_prev"][t]
        dh = dH[t] + dh_rec
        tc = np.tanh(c)
        da_o = dh * tc * o * (1.0 - o)       # output gate
        # c_t reaches the loss through h_t, the output gate's peephole and
        # (dc_rec) the next step
        dc = dh * o * (1.0 - tc * tc) + da_o * p_o + dc_rec
        da_i = dc * g * i * (1.0 - i)        # input gate
        da_f = dc * c_prev * f * (1.0 - f)   # forget gate
        da_g = dc * i * (1.0 - g * g)        # cell candidate
        da = np.concatenate([da_i, da_f, da_g, da_o])
        dA[t] = da
        dh_rec = W_hh.T @ da
        # c_{t-1} reaches the loss through the forget path and the two peepholes
        dc_rec = dc * f + da_i * p_i + da_f * p_f
    # Sums over the steps, each written as one product over the stored steps:
    # dW_hh = sum_t da_t h_{t-1}^T, dW_ih = sum_t da_t x_t^T, and the
    # peephole gradients sum_t da_i c_{t-1}, da_f c_{t-1}, da_o c_t.
    dW_hh = dA.T @ cache["h_prev"]
    dW_ih = dA.T @ X
    db = dA.sum(axis=0)
    dX = dA @ W_ih
    dp = np.concatenate([(dA[:, 0:H] * cache["c_prev"]).sum(axis=0),
                         (dA[:, H:2 * H] * cache["c_prev"]).sum(axis=0),
                         (dA[:, 3 * H:4 * H] * cache["c"]).sum(axis=0)])
    return dW_ih, dW_hh, db, dX, dp


def gru_dir_forward(W_ih, W_hh, b_ih, b_hh, X, d):
    L = X.shape[0]
    H = W_hh.shape[1]
    ax = X @ W_ih.T + b_ih
    Hs = np.zeros((L, H))
    cache = {k: np.zeros((L, H)) for k in ("r", "z", "n", "ahn", "h_prev")}
    h = np.zeros(H)
    for t in _time_order(L, d):
        ah = W_hh @ h + b_hh
        r = _sig(ax[t, 0:H] + ah[0:H])
        z = _sig(ax[t, H:2 * H] + ah[H:2 * H])
        n = np.tanh(ax[t, 2 * H:3 * H] + r * ah[2 * H:3 * H])
        cache["h_prev"][t] = h
        h = (1.0 - z) * n + z * h
        Hs[t] = h
        for k, v in (("r", r), ("z", z), ("n", n), ("ahn", ah[2 * H:3 * H])):
            cache[k][t] = v
    return Hs, cache


def gru_dir_backward(W_ih, W_hh, X, cache, dH, d):
    """Returns (dW_ih, dW_hh, db_ih, db_hh, dX)."""
    L = X.shape[0]
    H = W_hh.shape[1]
    dAx = np.zeros((L, 3 * H))   # gradient of the input pre-activations
    dAh = np.zeros((L, 3 * H))   # gradient of W_hh h + b_hh
    dh_rec = np.zeros(H)
    for t in reversed(list(_time_order(L, d))):
        r, z, n = cache["r"][t], cache["z"][t], cache["n"][t]
        ahn, h_prev = cache["ahn"][t], cache["h_prev"][t]
        dh = dH[t] + dh_rec
        dn = dh * (1.0 - z)
        dz = dh * (h_prev - n)
        dan = dn * (1.0 - n * n)
        dar = dan * ahn * r * (1.0 - r)
        daz = dz * z * (1.0 - z)
        dAx[t] = np.concatenate([dar, daz, dan])
        dAh[t] = np.concatenate([dar, daz, dan * r])
        dh_rec = W_hh.T @ dAh[t] + dh * z
    dW_hh = dAh.T @ cache["h_prev"]        # sum_t dAh_t h_{t-1}^T
    dW_ih = dAx.T @ X
    return dW_ih, dW_hh, dAx.sum(axis=0), dAh.sum(axis=0), dAx @ W_ih


def log_softmax(z):
    m = z.max(axis=-1, keepdims=True)
    return z - (m + np.log(np.exp(z - m).sum(axis=-1, keepdims=True)))


def forward_backward(m: Model, theta, seqs_x, seqs_y, need_grad=True, ctc_targets=None):
    """Loss and flat gradient for one mini-batch given as lists of per-sequence
    features [L_s, D] and labels [L_s].  Returns (loss, grad or None, outputs)
    where outputs holds the per-sequence top-layer activations.

    Per-frame loss: the mean over the batch's valid frames of the softmax
    cross-entropy of the frame's label.  With ctc_targets (one label string
    per sequence, classes 1..C-1; seqs_y is then not used): the mean over
    the batch's sequences of the CTC loss (oracle/ctc.py)."""
    from oracle import ctc
    p = unpack(m, theta)
    n_seq = len(seqs_x)
    G, H, dirs = m.gates, m.hidden, m.dirs
    n_valid = sum(int(len(y)) for y in seqs_y)
    grads = {k: np.zeros_like(v) for k, v in p.items()}
    loss = 0.0
    tops = []
    for X0, Y in zip(seqs_x, seqs_y):
        X0 = np.asarray(X0, np.float64)
        Y = np.asarray(Y, np.int64)
        L = X0.shape[0]
        inputs, caches = [X0], []
        for l in range(m.num_layers):
            outs = []
            for d in range(dirs):
                if m.is_lstm:
                    Hs, cache = lstm_dir_forward(p[("W_ih", l, d)], p[("W_hh", l, d)],
                                                 p[("b", l, d)], inputs[-1], d,
                                                 p.get(("p", l, d)))
                else:
                    Hs, cache = gru_dir_forward(p[("W_ih", l, d)], p[("W_hh", l, d)],
                                                p[("b_ih", l, d)], p[("b_hh", l, d)],
                                                inputs[-1], d)
                outs.append(Hs)
                caches.append(cache)
            inputs.append(np.concatenate(outs, axis=1))
        top = inputs[-1]
        tops.append(top)
        z = top @ p[("W_out", 0, 0)].T + p[("b_out", 0, 0)]
        if ctc_targets is not None:
            lc, gc = ctc.ctc_loss_grad(z, ctc_targets[len(tops) - 1])
            loss += lc / n_seq
            if not need_grad:
                continue
            dz = gc / n_seq
        else:
            logp = log_softmax(z)
            loss -= logp[np.arange(L), Y].sum() / n_valid
            if not need_grad:
                continue
            dz = np.exp(logp)
            dz[np.arange(L), Y] -= 1.0
            dz /= n_valid
        grads[("W_out", 0, 0)] += dz.T @ top
        grads[("b_out", 0, 0)] += dz.sum(axis=0)
        dIn = dz @ p[("W_out", 0, 0)]
        for l in range(m.num_layers - 1, -1, -1):
            X = inputs[l]
            dX = np.zeros_like(X)
            for d in range(dirs):
                cache = caches[l * dirs + d]
                dH = dIn[:, d * H:(d + 1) * H]
                if m.is_lstm:
                    gWi, gWh, gb, gX, gp = lstm_dir_backward(p[("W_ih", l, d)],
                                                             p[("W_hh", l, d)], X, cache, dH, d,
                                                             p.get(("p", l, d)))
                    grads[("b", l, d)] += gb
                    if m.cell == LSTM_PEEPHOLE:
                        grads[("p", l, d)] += gp
                else:
                    gWi, gWh, gbi, gbh, gX = gru_dir_backward(p[("W_ih", l, d)], p[("W_hh", l, d)],
                                                              X, cache, dH, d)
                    grads[("b_ih", l, d)] += gbi
                    grads[("b_hh", l, d)] += gbh
                grads[("W_ih", l, d)] += gWi
                grads[("W_hh", l, d)] += gWh
                dX += gX
            dIn = dX
    grad = pack(m, grads) if need_grad else None
    return float(loss), grad, tops


def sgd(theta, grad, lr):
    """Plain gradient-descent update theta - lr * grad (float64)."""
    return np.asarray(theta, np.float64) - lr * np.asarray(grad, np.float64)
