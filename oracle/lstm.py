"""LSTM layer with row-based dropout of hidden units, fixed per sequence, fp64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper applies the method to LSTM because the LSTM's work is matrix
multiplication (Sec. IV-C) but gives no equations. The reading used: the
hidden-unit mask m (a row pattern drawn once per sequence) removes dropped
units from the layer for the whole sequence. Their hidden and cell states are
held at zero, so the gate GEMMs shrink to the kept units (inputs x_t plus kept
h_{t-1}, outputs the four gates of kept units).

Gate order i, f, g, o; W = [W_ih | W_hh] stored as W[4H][I + H]:

    z_t = x_t W[:, :I]^T + (m * h_{t-1}) W[:, I:]^T + b
    i = sigmoid(z_i), f = sigmoid(z_f), g = tanh(z_g), o = sigmoid(z_o)
    c_t = m * (f * c_{t-1} + i * g)
    h_t = m * (o * tanh(c_t))

An optional input mask m_in (the hidden-unit pattern of the layer below, when
layers are stacked) removes dropped inputs the same way: the layer sees
x_t * m_in, so the input columns of dropped inputs take no part in any
product, and their entries of dX are 0.

Logical layout: X [T][B][I], h0 and c0 [B][H], outputs Hs [T][B][H].
Back-propagation through time takes dHs [T][B][H] (the derivative of the loss
with respect to every h_t) and optional extra derivatives dhT, dcT of the final
state, and returns dX, dW, db, dh0, dc0.
"""

import numpy as np


def _sigmoid(z):
    return 1.0 / (1.0 + np.exp(-z))


def lstm_forward(X, W, b, m, h0=None, c0=None, m_in=None):
    """Returns (Hs, hT, cT, cache)."""
    X = np.asarray(X, np.float64)
    if m_in is not None:
        X = X * np.asarray(m_in, np.float64)[None, None, :]
    W = np.asarray(W, np.float64)
    T, B, I = X.shape
    H = W.shape[0] // 4
    m = np.asarray(m, np.float64)
    h = np.zeros((B, H)) if h0 is None else np.asarray(h0, np.float64)
    c = np.zeros((B, H)) if c0 is None else np.asarray(c0, np.float64)
    bias = np.zeros(4 * H) if b is None else np.asarray(b, np.float64)
    Wx, Wh = W[:, :I], W[:, I:]
    Hs = np.zeros((T, B, H))
    cache = []
    for t in range(T):
        h_in = m[None, :] * h
        z = X[t] @ Wx.T + h_in @ Wh.T + bias[None, :]
        i = _sigmoid(z[:, 0:H])
        f = _sigmoid(z[:, H:2 * H])
        g = np.tanh(z[:, 2 * H:3 * H])
        o = _sigmoid(z[:, 3 * H:4 * H])
        c_prev = c
        c = m[None, :] * (f * c_prev + i * g)
        h = m[None, :] * (o * np.tanh(c))
        Hs[t] = h
        cache.append((h_in, c_prev, i, f, g, o, c))
    return Hs, h, c, cache


def lstm_backward(X, W, m, cache, dHs, dhT=None, dcT=None, m_in=None):
    """Manual back-propagation through time of ``lstm_forward``.

    Returns (dX, dW, db, dh0, dc0).
    """
    X = np.asarray(X, np.float64)
    if m_in is not None:
        X = X * np.asarray(m_in, np.float64)[None, None, :]
    W = np.asarray(W, np.float64)
    dHs = np.asarray(dHs, np.float64)
    T, B, I = X.shape
    H = W.shape[0] // 4
    m = np.asarray(m, np.float64)[None, :]
    Wx, Wh = W[:, :I], W[:, I:]
    dX = np.zeros_like(X)
    dW = np.zeros_like(W)
    db = np.zeros(4 * H)
    dh_next = np.zeros((B, H)) if dhT is None else np.asarray(dhT, np.float64).copy()
    dc_next = np.zeros((B, H)) if dcT is None else np.asarray(dcT, np.float64).copy()
    for t in range(T - 1, -1, -1):
        h_in, c_prev, i, f, g, o, c = cache[t]
        dh = m * (dHs[t] + dh_next)          # h_t = m * (o * tanh(c_t))
        tc = np.tanh(c)
        do = dh * tc
        dc = m * (dc_next + dh * o * (1.0 - tc * tc))   # c_t = m * (...)
        di = dc * g
        dg = dc * i
        df = dc * c_prev
        dz = np.concatenate([di * i * (1.0 - i),
                             df * f * (1.0 - f),
                             dg * (1.0 - g * g),
                             do * o * (1.0 - o)], axis=1)
        dX[t] = dz @ Wx
        dW[:, :I] += dz.T @ X[t]
        dW[:, I:] += dz.T @ h_in
        db += dz.sum(axis=0)
        dh_next = m * (dz @ Wh)              # the input was m * h_{t-1}
        dc_next = dc * f
    if m_in is not None:                     # the input was x_t * m_in
        dX = dX * np.asarray(m_in, np.float64)[None, None, :]
    return dX, dW, db, dh_next, dc_next
