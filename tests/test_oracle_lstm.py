"""Pins of the oracle's LSTM with hidden-unit row dropout (Sec. IV-C).

* dropout 0 equals torch.nn.LSTM (fp64, CPU): forward and autograd gradients;
* under a pattern, kept units equal a torch.nn.LSTM of hidden size |S| built
  from the gathered weights, dropped units stay at zero, and the manual
  back-propagation equals autograd through that compact model;
* finite differences on a tiny masked case.
"""
import numpy as np
import pytest
import torch

from oracle import lstm, patterns


def make(T, B, I, H, seed):
    rng = np.random.default_rng(seed)
    X = rng.uniform(-0.5, 0.5, size=(T, B, I))
    W = rng.uniform(-0.3, 0.3, size=(4 * H, I + H))
    b = rng.uniform(-0.3, 0.3, size=4 * H)
    h0 = rng.uniform(-0.5, 0.5, size=(B, H))
    c0 = rng.uniform(-0.5, 0.5, size=(B, H))
    dHs = rng.normal(size=(T, B, H))
    dhT = rng.normal(size=(B, H))
    dcT = rng.normal(size=(B, H))
    return X, W, b, h0, c0, dHs, dhT, dcT


def torch_lstm(X, W, b, h0, c0, dHs, dhT, dcT, I, H):
    """Run torch.nn.LSTM on the given (possibly compact) parameters; return
    outputs and gradients as numpy."""
    mod = torch.nn.LSTM(I, H).double()
    with torch.no_grad():
        mod.weight_ih_l0.copy_(torch.from_numpy(W[:, :I]))
        mod.weight_hh_l0.copy_(torch.from_numpy(W[:, I:]))
        mod.bias_ih_l0.copy_(torch.from_numpy(b))
        mod.bias_hh_l0.zero_()
    x = torch.from_numpy(X).requires_grad_(True)
    h = torch.from_numpy(h0)[None].clone().requires_grad_(True)
    c = torch.from_numpy(c0)[None].clone().requires_grad_(True)
    out, (hT, cT) = mod(x, (h, c))
    loss = (out * torch.from_numpy(dHs)).sum() + (hT[0] * torch.from_numpy(dhT)).sum() \
        + (cT[0] * torch.from_numpy(dcT)).sum()
    loss.backward()
    dW = np.concatenate([mod.weight_ih_l0.grad.numpy(), mod.weight_hh_l0.grad.numpy()], axis=1)
    return (out.detach().numpy(), hT[0].detach().numpy(), cT[0].detach().numpy(),
            x.grad.numpy(), dW, mod.bias_ih_l0.grad.numpy(), h.grad[0].numpy(), c.grad[0].numpy())


def test_rate_zero_equals_torch_lstm():
    T, B, I, H = 5, 3, 4, 6
    X, W, b, h0, c0, dHs, dhT, dcT = make(T, B, I, H, 0)
    m = patterns.row_mask(H, 1, 0)
    Hs, hT, cT, cache = lstm.lstm_forward(X, W, b, m, h0, c0)
    dX, dW, db, dh0, dc0 = lstm.lstm_backward(X, W, m, cache, dHs, dhT, dcT)
    ref = torch_lstm(X, W, b, h0, c0, dHs, dhT, dcT, I, H)
    for got, want in zip((Hs, hT, cT, dX, dW, db, dh0, dc0), ref):
        assert np.allclose(got, want, rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("period,offset", [(2, 0), (2, 1), (3, 2), (5, 4), (7, 6)])
def test_masked_equals_compact_torch_lstm(period, offset):
    T, B, I, H = 4, 2, 3, 10
    X, W, b, h0, c0, dHs, dhT, dcT = make(T, B, I, H, period * 10 + offset)
    S = patterns.row_kept_list(H, period, offset)
    m = patterns.row_mask(H, period, offset)
    Hs, hT, cT, cache = lstm.lstm_forward(X, W, b, m, h0, c0)
    dX, dW, db, dh0, dc0 = lstm.lstm_backward(X, W, m, cache, dHs, dhT, dcT)
    rows = [g * H + j for g in range(4) for j in S]
    Wc = np.concatenate([W[rows][:, :I], W[rows][:, [I + j for j in S]]], axis=1)
    r = torch_lstm(X, Wc, b[rows], h0[:, S], c0[:, S], dHs[:, :, S], dhT[:, S], dcT[:, S], I, len(S))
    dropped = [j for j in range(H) if j not in S]
    assert np.allclose(Hs[:, :, S], r[0], rtol=1e-12, atol=1e-13)
    assert not Hs[:, :, dropped].any() and not hT[:, dropped].any() and not cT[:, dropped].any()
    assert np.allclose(hT[:, S], r[1], rtol=1e-12, atol=1e-13)
    assert np.allclose(cT[:, S], r[2], rtol=1e-12, atol=1e-13)
    assert np.allclose(dX, r[3], rtol=1e-12, atol=1e-13)
    dWfull = np.zeros_like(W)
    cols = list(range(I)) + [I + j for j in S]
    dWfull[np.ix_(rows, cols)] = r[4]
    assert np.allclose(dW, dWfull, rtol=1e-12, atol=1e-13)
    dbfull = np.zeros(4 * H)
    dbfull[rows] = r[5]
    assert np.allclose(db, dbfull, rtol=1e-12, atol=1e-13)
    assert np.allclose(dh0[:, S], r[6], rtol=1e-12, atol=1e-13) and not dh0[:, dropped].any()
    assert np.allclose(dc0[:, S], r[7], rtol=1e-12, atol=1e-13) and not dc0[:, dropped].any()


@pytest.mark.parametrize("pin,ph", [((3, 1), (2, 0)), ((2, 0), (1, 0)), ((4, 3), (3, 2))])
def test_input_mask_equals_compact_torch_lstm(pin, ph):
    """An input pattern (the hidden pattern of the layer below): kept units
    equal a torch.nn.LSTM of input size |S_in| and hidden size |S| on the
    kept inputs, dX is torch's gradient at kept inputs and 0 at dropped ones,
    and the input columns of dropped inputs get no weight gradient."""
    T, B, I, H = 4, 2, 9, 6
    X, W, b, h0, c0, dHs, dhT, dcT = make(T, B, I, H, 31 + pin[0])
    Sin, S = patterns.row_kept_list(I, *pin), patterns.row_kept_list(H, *ph)
    m_in, m = patterns.row_mask(I, *pin), patterns.row_mask(H, *ph)
    Hs, hT, cT, cache = lstm.lstm_forward(X, W, b, m, h0, c0, m_in=m_in)
    dX, dW, db, dh0, dc0 = lstm.lstm_backward(X, W, m, cache, dHs, dhT, dcT, m_in=m_in)
    rows = [g * H + j for g in range(4) for j in S]
    cols = list(Sin) + [I + j for j in S]
    r = torch_lstm(X[:, :, Sin], W[np.ix_(rows, cols)], b[rows], h0[:, S], c0[:, S], dHs[:, :, S], dhT[:, S],
                   dcT[:, S], len(Sin), len(S))
    assert np.allclose(Hs[:, :, S], r[0], rtol=1e-12, atol=1e-13)
    assert np.allclose(dX[:, :, Sin], r[3], rtol=1e-12, atol=1e-13)
    dropped_in = [k for k in range(I) if k not in Sin]
    assert not dX[:, :, dropped_in].any()
    dWfull = np.zeros_like(W)
    dWfull[np.ix_(rows, cols)] = r[4]
    assert np.allclose(dW, dWfull, rtol=1e-12, atol=1e-13)
    assert np.allclose(db[rows], r[5], rtol=1e-12, atol=1e-13)
    assert np.allclose(dh0[:, S], r[6], rtol=1e-12, atol=1e-13)


def test_backward_is_the_derivative_of_forward():
    T, B, I, H = 3, 2, 2, 4
    X, W, b, h0, c0, dHs, dhT, dcT = make(T, B, I, H, 42)
    m = patterns.row_mask(H, 2, 1)

    def L(X_, W_, b_, h0_, c0_):
        Hs, hT, cT, _ = lstm.lstm_forward(X_, W_, b_, m, h0_, c0_)
        return float((Hs * dHs).sum() + (hT * dhT).sum() + (cT * dcT).sum())

    _, _, _, cache = lstm.lstm_forward(X, W, b, m, h0, c0)
    grads = lstm.lstm_backward(X, W, m, cache, dHs, dhT, dcT)
    args = [X, W, b, h0, c0]
    h = 1e-6
    for which, g in zip(range(5), grads):
        A = args[which]
        num = np.zeros_like(A)
        for idx in np.ndindex(A.shape):
            ap, am = list(args), list(args)
            ap[which], am[which] = A.copy(), A.copy()
            ap[which][idx] += h
            am[which][idx] -= h
            num[idx] = (L(*ap) - L(*am)) / (2 * h)
        assert np.allclose(num, g, rtol=1e-6, atol=1e-8)
