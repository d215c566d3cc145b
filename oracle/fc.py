"""Fully connected layer under a row-based dropout pattern, fp64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Conventional dropout multiplies a layer's output by a 0/1 mask in the forward
pass and its output derivative by the same mask in the backward pass
(Sec. II-C). Under a row-based pattern (Sec. III-A) the mask of a layer's
output neurons is m_out; the previous layer's pattern removes input features,
i.e. the columns of this layer's weight matrix, with mask m_in.

Logical math layout (the library stores activations feature-major, the
transposes of these):
    X [B][K] input, W [N][K] weights (one row per output neuron), b [N],
    Y [B][N] output, dY [B][N] output derivative.

Readings: the order is fully connected -> activation -> dropout (Sec. III-B,
last paragraph); dropped outputs are 0 (bias included); an explicit ``scale``
multiplies kept outputs (1 for a pure mask, 1/(1-p) for inverted dropout); the
ReLU derivative is taken from Y > 0, so that a backward pass fed the same
stored Y takes the same gating decisions as any other implementation.
"""

import numpy as np


def _relu(z):
    return np.where(z > 0.0, z, 0.0)


def fc_forward(X, W, bias, m_in, m_out, scale=1.0, act="none"):
    """Y = scale * m_out * act((X * m_in) W^T + b)."""
    X = np.asarray(X, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    Z = (X * m_in[None, :]) @ W.T
    if bias is not None:
        Z = Z + np.asarray(bias, dtype=np.float64)[None, :]
    A = _relu(Z) if act == "relu" else Z
    return scale * A * m_out[None, :]


def fc_output_grad(Y, dY, m_out, scale=1.0, act="none"):
    """G = scale * m_out * act'(.) * dY, with the ReLU derivative [Y > 0]."""
    dY = np.asarray(dY, dtype=np.float64)
    G = scale * dY * m_out[None, :]
    if act == "relu":
        G = G * (np.asarray(Y, dtype=np.float64) > 0.0)
    return G


def fc_backward(X, W, Y, dY, m_in, m_out, scale=1.0, act="none"):
    """Returns (dX, dW, db) of the masked layer.

    dX = m_in * (G W),  dW = (m_out outer m_in) * (G^T X),  db = sum_b G.
    """
    X = np.asarray(X, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    G = fc_output_grad(Y, dY, m_out, scale, act)
    dX = (G @ W) * m_in[None, :]
    dW = (G.T @ X) * np.outer(m_out, m_in)
    db = G.sum(axis=0)
    return dX, dW, db


def sgd_momentum(W, V, dW, m_out, m_in, lr, mu, b=None, Vb=None, db=None):
    """Momentum SGD restricted to the kept weights (the update of a training
    step around the method; Sec. IV trains with momentum SGD).

    Reading: a weight is updated in a step iff its output row and input column
    are both kept; dropped weights and their momentum stay as they are, and a
    bias entry is updated iff its row is kept. For the kept entries:
        V <- mu * V + dW,   W <- W - lr * V.
    Returns (W, V) or (W, V, b, Vb) as new fp64 arrays.
    """
    W = np.array(W, dtype=np.float64)
    V = np.array(V, dtype=np.float64)
    keep = np.outer(m_out, m_in) > 0
    Vn = mu * V + np.asarray(dW, dtype=np.float64)
    V = np.where(keep, Vn, V)
    W = np.where(keep, W - lr * V, W)
    if b is None:
        return W, V
    b = np.array(b, dtype=np.float64)
    Vb = np.array(Vb, dtype=np.float64)
    rows = np.asarray(m_out) > 0
    Vbn = mu * Vb + np.asarray(db, dtype=np.float64)
    Vb = np.where(rows, Vbn, Vb)
    b = np.where(rows, b - lr * Vb, b)
    return W, V, b, Vb
