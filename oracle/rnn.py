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
The sequences of a batch run side by side, each over its own length: at
step k every sequence longer than k advances one frame (frame k, or its
frame L - 1 - k in the reverse direction) from its own state.  Frames past
a sequence's length are padding that takes no part in anything.

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


def _steps(lengths, d: int):
    """The recurrence's steps over a batch of sequences run side by side:
    at step k (k = 0 .. max length - 1) every sequence still running
    (k < L_b) advances by one frame -- frame k forward, frame L_b - 1 - k in
    the reverse direction.  Yields (rows, frames) per step."""
    lengths = np.asarray(lengths)
    for k in range(int(lengths.max())):
        rows = np.nonzero(lengths > k)[0]
        yield rows, (np.full(rows.size, k) if d == 0 else lengths[rows] - 1 - k)


def valid_mask(lengths, T: int) -> np.ndarray:
    """[B, T] booleans: frame t of sequence b exists (t < L_b)."""
    return np.arange(T)[None, :] < np.asarray(lengths)[:, None]


def lstm_dir_forward(W_ih, W_hh, b, X, lengths, d, peep=None):
    """One direction of one LSTM layer over a batch of sequences given as a
    padded array X [B, T, D_in] (frames t >= L_b are never used) with
    lengths [B]; every sequence runs its own recurrence from a zero state
    (see _steps).  `peep` = [p_i ; p_f ; p_o] (3H) for the peephole cell,
    else None.  Returns (Hseq [B, T, H] with zero pad frames, cache)."""
    B, T = X.shape[0], X.shape[1]
    H = W_hh.shape[1]
    p_i, p_f, p_o = (np.zeros(H),) * 3 if peep is None else np.reshape(peep, (3, H))
    Hs = np.zeros((B, T, H))
    cache = {k: np.zeros((B, T, H)) for k in ("i", "f", "g", "o", "c", "c_prev", "h_prev")}
    h = np.zeros((B, H))
    c = np.zeros((B, H))
    for rows, fr in _steps(lengths, d):
        a = X[rows, fr] @ W_ih.T + b + h[rows] @ W_hh.T
        cp = c[rows]
        i = _sig(a[:, 0:H] + p_i * cp)
        f = _sig(a[:, H:2 * H] + p_f * cp)
        g = np.tanh(a[:, 2 * H:3 * H])
        cache["h_prev"][rows, fr] = h[rows]
        cache["c_prev"][rows, fr] = cp
        cn = f * cp + i * g
        o = _sig(a[:, 3 * H:4 * H] + p_o * cn)
        hn = o * np.tanh(cn)
        c[rows] = cn
        h[rows] = hn
        Hs[rows, fr] = hn
        for k, v in (("i", i), ("f", f), ("g", g), ("o", o), ("c", cn)):
            cache[k][rows, fr] = v
    return Hs, cache


def lstm_dir_backward(W_ih, W_hh, X, lengths, cache, dH, d, peep=None):
    """Reverse-mode pass of ``lstm_dir_forward`` given dLoss/dh = dH
    [B, T, H] (zero on pad frames).  Returns (dW_ih, dW_hh, db, dX
    [B, T, D_in], dpeep); dpeep (3H) is zero without peepholes."""
    B, T = X.shape[0], X.shape[1]
    H = W_hh.shape[1]
    p_i, p_f, p_o = (np.zeros(H),) * 3 if peep is None else np.reshape(peep, (3, H))
    dA = np.zeros((B, T, 4 * H))
    dh_rec = np.zeros((B, H))  # gradient reaching h_t through the next step's W_hh
    dc_rec = np.zeros((B, H))  # gradient reaching c_t through the next step's gates
    for rows, fr in reversed(list(_steps(lengths, d))):
        i, f, g, o = (cache[k][rows, fr] for k in ("i", "f", "g", "o"))
        c, c_prev = cache["c"][rows, fr], cache["c_prev"][rows, fr]
        dh = dH[rows, fr] + dh_rec[rows]
        tc = np.tanh(c)
        da_o = dh * tc * o * (1.0 - o)       # output gate
        # c_t reaches the loss through h_t, the output gate's peephole and
        # (dc_rec) the next step
        dc = dh * o * (1.0 - tc * tc) + da_o * p_o + dc_rec[rows]
        da_i = dc * g * i * (1.0 - i)        # input gate
        da_f = dc * c_prev * f * (1.0 - f)   # forget gate
        da_g = dc * i * (1.0 - g * g)        # cell candidate
        da = np.concatenate([da_i, da_f, da_g, da_o], axis=1)
        dA[rows, fr] = da
        dh_rec[rows] = da @ W_hh
        # c_{t-1} reaches the loss through the forget path and the two peepholes
        dc_rec[rows] = dc * f + da_i * p_i + da_f * p_f
    # Sums over every valid frame, each written as one product:
    # dW_hh = sum da_t h_{t-1}^T, dW_ih = sum da_t x_t^T, and the peephole
    # gradients sum da_i c_{t-1}, da_f c_{t-1}, da_o c_t.
    M = valid_mask(lengths, T)
    dAv = dA[M]
    dW_hh = dAv.T @ cache["h_prev"][M]
    dW_ih = dAv.T @ X[M]
    db = dAv.sum(axis=0)
    dX = dA @ W_ih
    dp = np.concatenate([(dAv[:, 0:H] * cache["c_prev"][M]).sum(axis=0),
                         (dAv[:, H:2 * H] * cache["c_prev"][M]).sum(axis=0),
                         (dAv[:, 3 * H:4 * H] * cache["c"][M]).sum(axis=0)])
    return dW_ih, dW_hh, db, dX, dp


def gru_dir_forward(W_ih, W_hh, b_ih, b_hh, X, lengths, d):
    """As lstm_dir_forward for the GRU cell."""
    B, T = X.shape[0], X.shape[1]
    H = W_hh.shape[1]
    Hs = np.zeros((B, T, H))
    cache = {k: np.zeros((B, T, H)) for k in ("r", "z", "n", "ahn", "h_prev")}
    h = np.zeros((B, H))
    for rows, fr in _steps(lengths, d):
        hp = h[rows]
        ax = X[rows, fr] @ W_ih.T + b_ih
        ah = hp @ W_hh.T + b_hh
        r = _sig(ax[:, 0:H] + ah[:, 0:H])
        z = _sig(ax[:, H:2 * H] + ah[:, H:2 * H])
        n = np.tanh(ax[:, 2 * H:3 * H] + r * ah[:, 2 * H:3 * H])
        cache["h_prev"][rows, fr] = hp
        hn = (1.0 - z) * n + z * hp
        h[rows] = hn
        Hs[rows, fr] = hn
        for k, v in (("r", r), ("z", z), ("n", n), ("ahn", ah[:, 2 * H:3 * H])):
            cache[k][rows, fr] = v
    return Hs, cache


def gru_dir_backward(W_ih, W_hh, X, lengths, cache, dH, d):
    """Returns (dW_ih, dW_hh, db_ih, db_hh, dX [B, T, D_in])."""
    B, T = X.shape[0], X.shape[1]
    H = W_hh.shape[1]
    dAx = np.zeros((B, T, 3 * H))   # gradient of the input pre-activations
    dAh = np.zeros((B, T, 3 * H))   # gradient of W_hh h + b_hh
    dh_rec = np.zeros((B, H))
    for rows, fr in reversed(list(_steps(lengths, d))):
        r, z, n = cache["r"][rows, fr], cache["z"][rows, fr], cache["n"][rows, fr]
        ahn, h_prev = cache["ahn"][rows, fr], cache["h_prev"][rows, fr]
        dh = dH[rows, fr] + dh_rec[rows]
        dn = dh * (1.0 - z)
        dz = dh * (h_prev - n)
        dan = dn * (1.0 - n * n)
        dar = dan * ahn * r * (1.0 - r)
        daz = dz * z * (1.0 - z)
        dAx[rows, fr] = np.concatenate([dar, daz, dan], axis=1)
        dah = np.concatenate([dar, daz, dan * r], axis=1)
        dAh[rows, fr] = dah
        dh_rec[rows] = dah @ W_hh + dh * z
    M = valid_mask(lengths, T)
    dW_hh = dAh[M].T @ cache["h_prev"][M]        # sum dAh_t h_{t-1}^T
    dW_ih = dAx[M].T @ X[M]
    return dW_ih, dW_hh, dAx[M].sum(axis=0), dAh[M].sum(axis=0), dAx @ W_ih


def log_softmax(z):
    m = z.max(axis=-1, keepdims=True)
    return z - (m + np.log(np.exp(z - m).sum(axis=-1, keepdims=True)))


def forward_backward(m: Model, theta, seqs_x, seqs_y, need_grad=True, ctc_targets=None):
    """Loss and flat gradient for one mini-batch given as lists of per-sequence
    features [L_s, D] and labels [L_s].  Returns (loss, grad or None, outputs)
    where outputs holds the per-sequence top-layer activations [L_s, H_top].

    The sequences run side by side, each over its own length (see _steps);
    frames past a sequence's length take no part in anything.
    Per-frame loss: the mean over the batch's valid frames of the softmax
    cross-entropy of the frame's label.  With ctc_targets (one label string
    per sequence, classes 1..C-1; seqs_y is then not used): the mean over
    the batch's sequences of the CTC loss (oracle/ctc.py)."""
    from oracle import ctc
    p = unpack(m, theta)
    n_seq = len(seqs_x)
    H, dirs = m.hidden, m.dirs
    lengths = np.array([len(x) for x in seqs_x], np.int64)
    if n_seq == 0 or lengths.min() < 1:
        raise ValueError("every sequence needs at least one frame")
    T = int(lengths.max())
    X0 = np.zeros((n_seq, T, m.input_dim))
    for b, x in enumerate(seqs_x):
        X0[b, :lengths[b]] = np.asarray(x, np.float64)
    M = valid_mask(lengths, T)
    n_valid = int(lengths.sum())
    grads = {k: np.zeros_like(v) for k, v in p.items()}
    inputs, caches = [X0], []
    for l in range(m.num_layers):
        outs = []
        for d in range(dirs):
            if m.is_lstm:
                Hs, cache = lstm_dir_forward(p[("W_ih", l, d)], p[("W_hh", l, d)],
                                             p[("b", l, d)], inputs[-1], lengths, d,
                                             p.get(("p", l, d)))
            else:
                Hs, cache = gru_dir_forward(p[("W_ih", l, d)], p[("W_hh", l, d)],
                                            p[("b_ih", l, d)], p[("b_hh", l, d)],
                                            inputs[-1], lengths, d)
            outs.append(Hs)
            caches.append(cache)
        inputs.append(np.concatenate(outs, axis=2))
    top = inputs[-1]
    tops = [top[b, :lengths[b]] for b in range(n_seq)]
    z = top @ p[("W_out", 0, 0)].T + p[("b_out", 0, 0)]       # [B, T, C]
    dz = np.zeros_like(z)
    if ctc_targets is not None:
        loss = 0.0
        for b in range(n_seq):
            lc, gc = ctc.ctc_loss_grad(z[b, :lengths[b]], ctc_targets[b])
            loss += lc / n_seq
            dz[b, :lengths[b]] = gc / n_seq
    else:
        Y = np.zeros((n_seq, T), np.int64)
        for b, y in enumerate(seqs_y):
            Y[b, :lengths[b]] = np.asarray(y, np.int64)
        logp = log_softmax(z[M])                                  # valid frames only
        picked = logp[np.arange(n_valid), Y[M]]
        loss = -picked.sum() / n_valid
        g = np.exp(logp)
        g[np.arange(n_valid), Y[M]] -= 1.0
        dz[M] = g / n_valid
    if not need_grad:
        return float(loss), None, tops
    grads[("W_out", 0, 0)] += dz[M].T @ top[M]
    grads[("b_out", 0, 0)] += dz[M].sum(axis=0)
    dIn = dz @ p[("W_out", 0, 0)]                                  # zero on pad frames
    for l in range(m.num_layers - 1, -1, -1):
        X = inputs[l]
        dX = np.zeros_like(X)
        for d in range(dirs):
            cache = caches[l * dirs + d]
            dH = dIn[:, :, d * H:(d + 1) * H]
            if m.is_lstm:
                gWi, gWh, gb, gX, gp = lstm_dir_backward(p[("W_ih", l, d)], p[("W_hh", l, d)],
                                                         X, lengths, cache, dH, d,
                                                         p.get(("p", l, d)))
                grads[("b", l, d)] += gb
                if m.cell == LSTM_PEEPHOLE:
                    grads[("p", l, d)] += gp
            else:
                gWi, gWh, gbi, gbh, gX = gru_dir_backward(p[("W_ih", l, d)], p[("W_hh", l, d)],
                                                          X, lengths, cache, dH, d)
                grads[("b_ih", l, d)] += gbi
                grads[("b_hh", l, d)] += gbh
            grads[("W_ih", l, d)] += gWi
            grads[("W_hh", l, d)] += gWh
            dX += gX
        dIn = dX * M[:, :, None]
    return float(loss), pack(m, grads), tops


def sgd(theta, grad, lr):
    """Plain gradient-descent update theta - lr * grad (float64)."""
    return np.asarray(theta, np.float64) - lr * np.asarray(grad, np.float64)
