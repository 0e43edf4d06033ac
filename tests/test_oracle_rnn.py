"""Pins of the float64 recurrent-model oracle.

Forward values are pinned to closed forms of the LSTM cell and to PyTorch's
own CPU LSTM/GRU in float64 (an independent library implementation with the
same gate equations); gradients to central finite differences and to
autograd through that library model; the loss to its value at zero output
weights."""
import math

import numpy as np
import pytest
import torch

from oracle import rnn



def _rand_batch(rng, lengths, D, C):
    xs = [rng.standard_normal((L, D)) for L in lengths]
    ys = [rng.integers(0, C, L) for L in lengths]
    return xs, ys


def _torch_model(m, theta):
    """Builds torch.nn.LSTM/GRU + Linear holding the oracle's parameters."""
    p = rnn.unpack(m, theta)
    cls = torch.nn.LSTM if m.cell == rnn.LSTM else torch.nn.GRU
    net = cls(m.input_dim, m.hidden, m.num_layers, bidirectional=bool(m.bidirectional),
              dtype=torch.float64)
    lin = torch.nn.Linear(m.hidden * m.dirs, m.num_classes, dtype=torch.float64)
    with torch.no_grad():
        for l in range(m.num_layers):
            for d in range(m.dirs):
                sfx = f"_l{l}" + ("_reverse" if d else "")
                getattr(net, "weight_ih" + sfx).copy_(torch.tensor(p[("W_ih", l, d)]))
                getattr(net, "weight_hh" + sfx).copy_(torch.tensor(p[("W_hh", l, d)]))
                if m.cell == rnn.LSTM:
                    getattr(net, "bias_ih" + sfx).copy_(torch.tensor(p[("b", l, d)]))
                    getattr(net, "bias_hh" + sfx).zero_()
                else:
                    getattr(net, "bias_ih" + sfx).copy_(torch.tensor(p[("b_ih", l, d)]))
                    getattr(net, "bias_hh" + sfx).copy_(torch.tensor(p[("b_hh", l, d)]))
        lin.weight.copy_(torch.tensor(p[("W_out", 0, 0)]))
        lin.bias.copy_(torch.tensor(p[("b_out", 0, 0)]))
    return net, lin


def _torch_loss_grad(m, theta, xs, ys, ctc_targets=None):
    net, lin = _torch_model(m, theta)
    lengths = torch.tensor([len(y) for y in ys])
    padded = torch.nn.utils.rnn.pad_sequence([torch.tensor(x) for x in xs])
    packed = torch.nn.utils.rnn.pack_padded_sequence(padded, lengths, enforce_sorted=False)
    out, _ = net(packed)
    out, _ = torch.nn.utils.rnn.pad_packed_sequence(out)
    tops = [out[:L, b] for b, L in enumerate(lengths.tolist())]
    top = torch.cat(tops)
    if ctc_targets is None:
        y = torch.cat([torch.tensor(np.asarray(v)) for v in ys])
        loss = torch.nn.functional.cross_entropy(lin(top), y, reduction="mean")
    else:
        # CTC, mean over sequences: torch's ctc_loss summed, divided by the count
        lp = torch.nn.utils.rnn.pad_sequence([torch.log_softmax(lin(t), dim=1) for t in tops])
        tg = torch.cat([torch.tensor(np.asarray(t), dtype=torch.long) for t in ctc_targets])
        tl = torch.tensor([len(t) for t in ctc_targets])
        loss = torch.nn.functional.ctc_loss(lp, tg, lengths, tl, blank=0, reduction="sum",
                                            zero_infinity=False) / len(xs)
    loss.backward()
    grads = {}
    for l in range(m.num_layers):
        for d in range(m.dirs):
            sfx = f"_l{l}" + ("_reverse" if d else "")
            grads[("W_ih", l, d)] = getattr(net, "weight_ih" + sfx).grad.numpy()
            grads[("W_hh", l, d)] = getattr(net, "weight_hh" + sfx).grad.numpy()
            if m.cell == rnn.LSTM:
                grads[("b", l, d)] = getattr(net, "bias_ih" + sfx).grad.numpy()
            else:
                grads[("b_ih", l, d)] = getattr(net, "bias_ih" + sfx).grad.numpy()
                grads[("b_hh", l, d)] = getattr(net, "bias_hh" + sfx).grad.numpy()
    grads[("W_out", 0, 0)] = lin.weight.grad.numpy()
    grads[("b_out", 0, 0)] = lin.bias.grad.numpy()
    return loss.item(), rnn.pack(m, grads), [t.detach().numpy() for t in tops]


MODELS = [
    rnn.Model(rnn.LSTM, 1, 0, 3, 5, 4),
    rnn.Model(rnn.LSTM, 2, 0, 3, 4, 5),
    rnn.Model(rnn.LSTM, 2, 1, 3, 4, 5),
    rnn.Model(rnn.GRU, 2, 0, 3, 4, 5),
    rnn.Model(rnn.GRU, 2, 1, 2, 3, 4),
]


@pytest.mark.parametrize("mi", range(len(MODELS)))
def test_matches_torch_float64(mi):
    m = MODELS[mi]
    rng = np.random.default_rng(mi)
    theta = rng.uniform(-0.5, 0.5, rnn.param_count(m))
    lengths = [7, 5, 5, 2, 1]
    xs, ys = _rand_batch(rng, lengths, m.input_dim, m.num_classes)
    loss, grad, tops = rnn.forward_backward(m, theta, xs, ys)
    tloss, tgrad, ttops = _torch_loss_grad(m, theta, xs, ys)
    for a, b in zip(tops, ttops):
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)
    assert abs(loss - tloss) < 1e-12
    np.testing.assert_allclose(grad, tgrad, rtol=0, atol=1e-10)


def _rand_targets(rng, lengths, C):
    return [rng.integers(1, C, max(1, L // 3)) for L in lengths]


@pytest.mark.parametrize("mi", range(len(MODELS)))
def test_ctc_matches_torch_float64(mi):
    """The model with the CTC loss against PyTorch's LSTM/GRU + ctc_loss."""
    m = MODELS[mi]
    rng = np.random.default_rng(40 + mi)
    theta = rng.uniform(-0.5, 0.5, rnn.param_count(m))
    lengths = [9, 7, 7, 3, 1]
    xs, ys = _rand_batch(rng, lengths, m.input_dim, m.num_classes)
    tg = _rand_targets(rng, lengths, m.num_classes)
    loss, grad, _ = rnn.forward_backward(m, theta, xs, ys, ctc_targets=tg)
    tloss, tgrad, _ = _torch_loss_grad(m, theta, xs, ys, ctc_targets=tg)
    assert abs(loss - tloss) < 1e-11 * abs(tloss)
    np.testing.assert_allclose(grad, tgrad, rtol=0, atol=1e-10)


@pytest.mark.parametrize("mi", [0, 3])
def test_ctc_finite_differences(mi):
    m = MODELS[mi]
    rng = np.random.default_rng(50 + mi)
    theta = rng.uniform(-0.5, 0.5, rnn.param_count(m))
    lengths = [6, 4, 2]
    xs, ys = _rand_batch(rng, lengths, m.input_dim, m.num_classes)
    tg = _rand_targets(rng, lengths, m.num_classes)
    _, grad, _ = rnn.forward_backward(m, theta, xs, ys, ctc_targets=tg)
    h = 1e-6
    fd = np.zeros_like(theta)
    for k in range(theta.size):
        tp = theta.copy(); tp[k] += h
        tm = theta.copy(); tm[k] -= h
        fd[k] = (rnn.forward_backward(m, tp, xs, ys, False, tg)[0]
                 - rnn.forward_backward(m, tm, xs, ys, False, tg)[0]) / (2 * h)
    err = np.abs(fd - grad) / np.maximum(np.abs(grad), 1e-3)
    assert err.max() < 1e-6, err.max()


@pytest.mark.parametrize("mi", range(len(MODELS)))
def test_finite_differences(mi):
    m = MODELS[mi]
    rng = np.random.default_rng(10 + mi)
    theta = rng.uniform(-0.5, 0.5, rnn.param_count(m))
    lengths = [6, 4, 1]
    xs, ys = _rand_batch(rng, lengths, m.input_dim, m.num_classes)
    _, grad, _ = rnn.forward_backward(m, theta, xs, ys)
    h = 1e-6
    fd = np.zeros_like(theta)
    for k in range(theta.size):
        tp = theta.copy(); tp[k] += h
        tm = theta.copy(); tm[k] -= h
        fd[k] = (rnn.forward_backward(m, tp, xs, ys, need_grad=False)[0]
                 - rnn.forward_backward(m, tm, xs, ys, need_grad=False)[0]) / (2 * h)
    err = np.abs(fd - grad) / np.maximum(np.abs(grad), 1e-3)
    assert err.max() < 1e-6, err.max()


def _lstm_bias_only(H, b_g, b_f=0.0):
    m = rnn.Model(rnn.LSTM, 1, 0, 2, H, 3)
    p = {k: np.zeros(s) for k, s in rnn.param_layout(m)}
    p[("b", 0, 0)][2 * H:3 * H] = b_g
    p[("b", 0, 0)][H:2 * H] = b_f
    return m, rnn.pack(m, p)


@pytest.mark.parametrize("T", [1, 2, 17, 4000])
def test_closed_form_half_gates(T):
    # All weights zero, only the cell-candidate bias b: i = f = o = 1/2,
    # c_t = tanh(b) * (1 - 2^-(t+1)), h_t = tanh(c_t) / 2.
    H = 3
    b = np.array([0.3, -1.2, 2.0])
    m, theta = _lstm_bias_only(H, b)
    x = np.random.default_rng(0).standard_normal((T, 2))
    _, _, tops = rnn.forward_backward(m, theta, [x], [np.zeros(T, int)], need_grad=False)
    t = np.arange(T)[:, None]
    c = np.tanh(b)[None, :] * (1.0 - 2.0 ** (-(t + 1.0)))
    np.testing.assert_allclose(tops[0], 0.5 * np.tanh(c), rtol=0, atol=1e-15)


@pytest.mark.parametrize("T", [1, 5, 4000])
def test_closed_form_running_sum(T):
    # Forget-gate bias 40 makes f == 1.0 exactly in float64, so the cell is the
    # running sum c_t = (t+1) * tanh(b) / 2 and h_t = tanh(c_t) / 2.
    H = 2
    b = np.array([0.001, -0.0005])
    m, theta = _lstm_bias_only(H, b, b_f=40.0)
    x = np.zeros((T, 2))
    _, _, tops = rnn.forward_backward(m, theta, [x], [np.zeros(T, int)], need_grad=False)
    t = np.arange(T)[:, None]
    c = (t + 1.0) * 0.5 * np.tanh(b)[None, :]
    np.testing.assert_allclose(tops[0], 0.5 * np.tanh(c), rtol=1e-13, atol=0)


def test_loss_at_zero_output_weights():
    m = rnn.Model(rnn.LSTM, 1, 1, 3, 4, 7)
    rng = np.random.default_rng(3)
    p = {k: rng.uniform(-0.3, 0.3, s) for k, s in rnn.param_layout(m)}
    p[("W_out", 0, 0)][:] = 0
    p[("b_out", 0, 0)][:] = 0
    theta = rnn.pack(m, p)
    xs, ys = _rand_batch(rng, [5, 3], 3, 7)
    loss, grad, _ = rnn.forward_backward(m, theta, xs, ys)
    assert abs(loss - math.log(7)) < 1e-14
    g = rnn.unpack(m, grad)
    y = np.concatenate(ys)
    expect = (np.full(7, 1.0 / 7) * len(y) - np.bincount(y, minlength=7)) / len(y)
    np.testing.assert_allclose(g[("b_out", 0, 0)], expect, atol=1e-15)
    for (kind, _, _), v in g.items():
        if kind not in ("W_out", "b_out"):
            assert np.all(v == 0)


def test_batch_invariances():
    m = rnn.Model(rnn.LSTM, 2, 1, 3, 4, 5)
    rng = np.random.default_rng(4)
    theta = rng.uniform(-0.5, 0.5, rnn.param_count(m))
    xs, ys = _rand_batch(rng, [6, 3, 3, 1], 3, 5)
    loss, grad, _ = rnn.forward_backward(m, theta, xs, ys)
    perm = [2, 0, 3, 1]
    loss_p, grad_p, _ = rnn.forward_backward(m, theta, [xs[i] for i in perm], [ys[i] for i in perm])
    assert abs(loss - loss_p) < 1e-14
    np.testing.assert_allclose(grad, grad_p, atol=1e-15)
    # splitting the batch: N-weighted sums add up
    l1, g1, _ = rnn.forward_backward(m, theta, xs[:2], ys[:2])
    l2, g2, _ = rnn.forward_backward(m, theta, xs[2:], ys[2:])
    n1, n2 = 9, 4
    assert abs(loss * 13 - (l1 * n1 + l2 * n2)) < 1e-12
    np.testing.assert_allclose(grad * 13, g1 * n1 + g2 * n2, atol=1e-13)


def test_sgd_exact():
    theta = np.array([1.0, -2.0, 0.5])
    g = np.array([0.25, 1.0, -4.0])
    np.testing.assert_array_equal(rnn.sgd(theta, g, 0.5), [0.875, -2.5, 2.5])


def test_param_count_formula():
    m = rnn.Model(rnn.LSTM, 3, 1, 8, 256, 80)
    assert rnn.param_count(m) == 3733584
    m = rnn.Model(rnn.GRU, 2, 0, 8, 384, 80)
    assert rnn.param_count(m) == 1371728


# ------------------------------------------------------------ peephole LSTM

PEEP_MODELS = [
    rnn.Model(rnn.LSTM_PEEPHOLE, 1, 0, 3, 4, 5),
    rnn.Model(rnn.LSTM_PEEPHOLE, 2, 1, 2, 3, 4),
]


def _sig(v):
    return 1.0 / (1.0 + math.exp(-v))


def test_peephole_closed_form_two_steps():
    """Weights zero, biases and peepholes set: the first two steps worked out
    by hand.  Step 0 starts from c = 0, so only the output gate's peephole
    (which sees the new cell state) acts; step 1 brings in p_i and p_f through
    c_0.  Distinct p_i, p_f, p_o catch a swapped or mis-timed peephole."""
    H = 2
    m = rnn.Model(rnn.LSTM_PEEPHOLE, 1, 0, 2, H, 3)
    p = {k: np.zeros(s) for k, s in rnn.param_layout(m)}
    b_i, b_f, b_g, b_o = [0.4, -0.3], [0.2, 0.9], [1.1, -0.7], [-0.5, 0.3]
    p_i, p_f, p_o = [1.5, -0.8], [-1.2, 0.6], [2.0, -2.5]
    p[("b", 0, 0)][:] = np.concatenate([b_i, b_f, b_g, b_o])
    p[("p", 0, 0)][:] = np.concatenate([p_i, p_f, p_o])
    theta = rnn.pack(m, p)
    x = np.random.default_rng(2).standard_normal((2, 2))
    _, _, tops = rnn.forward_backward(m, theta, [x], [np.zeros(2, int)], need_grad=False)
    for u in range(H):
        c0 = _sig(b_i[u]) * math.tanh(b_g[u])
        h0 = _sig(b_o[u] + p_o[u] * c0) * math.tanh(c0)
        c1 = _sig(b_f[u] + p_f[u] * c0) * c0 + _sig(b_i[u] + p_i[u] * c0) * math.tanh(b_g[u])
        h1 = _sig(b_o[u] + p_o[u] * c1) * math.tanh(c1)
        np.testing.assert_allclose(tops[0][:, u], [h0, h1], rtol=1e-15, atol=0)


@pytest.mark.parametrize("ctc", [False, True])
def test_peephole_zero_is_the_plain_lstm(ctc):
    """With p = 0 the peephole cell is the plain LSTM: the outputs, the loss
    and every shared gradient block agree exactly."""
    mp = rnn.Model(rnn.LSTM_PEEPHOLE, 2, 1, 3, 4, 5)
    m0 = rnn.Model(rnn.LSTM, 2, 1, 3, 4, 5)
    rng = np.random.default_rng(7)
    p0 = {k: rng.uniform(-0.5, 0.5, s) for k, s in rnn.param_layout(m0)}
    pp = dict(p0)
    for l in range(2):
        for d in range(2):
            pp[("p", l, d)] = np.zeros(12)
    lengths = [6, 4, 4, 1]
    xs, ys = _rand_batch(rng, lengths, 3, 5)
    tg = _rand_targets(rng, lengths, 5) if ctc else None
    l0, g0, t0 = rnn.forward_backward(m0, rnn.pack(m0, p0), xs, ys, ctc_targets=tg)
    lp, gp, tp = rnn.forward_backward(mp, rnn.pack(mp, pp), xs, ys, ctc_targets=tg)
    assert l0 == lp
    for a, b in zip(t0, tp):
        np.testing.assert_array_equal(a, b)
    g0, gp = rnn.unpack(m0, g0), rnn.unpack(mp, gp)
    for k in g0:
        np.testing.assert_array_equal(g0[k], gp[k])


@pytest.mark.parametrize("mi", range(len(PEEP_MODELS)))
@pytest.mark.parametrize("ctc", [False, True])
def test_peephole_finite_differences(mi, ctc):
    m = PEEP_MODELS[mi]
    rng = np.random.default_rng(60 + mi)
    theta = rng.uniform(-0.8, 0.8, rnn.param_count(m))
    lengths = [6, 4, 1]
    xs, ys = _rand_batch(rng, lengths, m.input_dim, m.num_classes)
    tg = _rand_targets(rng, lengths, m.num_classes) if ctc else None
    _, grad, _ = rnn.forward_backward(m, theta, xs, ys, ctc_targets=tg)
    h = 1e-6
    fd = np.zeros_like(theta)
    for k in range(theta.size):
        tp = theta.copy(); tp[k] += h
        tm = theta.copy(); tm[k] -= h
        fd[k] = (rnn.forward_backward(m, tp, xs, ys, False, tg)[0]
                 - rnn.forward_backward(m, tm, xs, ys, False, tg)[0]) / (2 * h)
    err = np.abs(fd - grad) / np.maximum(np.abs(grad), 1e-3)
    assert err.max() < 1e-6, err.max()
    # the peephole blocks carry gradient (a dropped term would leave them 0)
    g = rnn.unpack(m, grad)
    assert all(np.abs(v).max() > 1e-4 for (kind, _, _), v in g.items() if kind == "p")


def test_peephole_param_count():
    m = rnn.Model(rnn.LSTM_PEEPHOLE, 2, 0, 8, 128, 80)
    plain = rnn.Model(rnn.LSTM, 2, 0, 8, 128, 80)
    assert rnn.param_count(m) == rnn.param_count(plain) + 2 * 3 * 128
