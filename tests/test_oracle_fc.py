"""Pins of the oracle's FC layer under a row pattern (Sec. II-C, Sec. III-A).

* brute force: the definition evaluated element by element in pure Python;
* compaction: gathering the kept rows/columns, multiplying the compact
  matrices and scattering back gives bitwise the masked dense result on
  integer-valued inputs (fp64 is exact there), for every (period, offset);
* finite differences of the forward pass give the backward pass.
"""
import itertools

import numpy as np
import pytest

from oracle import fc, patterns


def brute_forward(X, W, b, kin, kout, scale, act):
    B, K = len(X), len(X[0])
    N = len(W)
    Y = [[0.0] * N for _ in range(B)]
    for s in range(B):
        for n in range(N):
            if n not in kout:
                continue
            z = b[n] if b is not None else 0.0
            for k in range(K):
                if k in kin:
                    z += X[s][k] * W[n][k]
            if act == "relu":
                z = max(z, 0.0)
            Y[s][n] = scale * z
    return np.array(Y)


def brute_backward(X, W, Y, dY, kin, kout, scale, act):
    B, K, N = len(X), len(X[0]), len(W)
    G = [[0.0] * N for _ in range(B)]
    for s in range(B):
        for n in range(N):
            if n in kout and (act != "relu" or Y[s][n] > 0):
                G[s][n] = scale * dY[s][n]
    dX = [[sum(G[s][n] * W[n][k] for n in range(N)) if k in kin else 0.0
           for k in range(K)] for s in range(B)]
    dW = [[sum(G[s][n] * X[s][k] for s in range(B)) if (n in kout and k in kin) else 0.0
           for k in range(K)] for n in range(N)]
    db = [sum(G[s][n] for s in range(B)) for n in range(N)]
    return np.array(dX), np.array(dW), np.array(db)


@pytest.mark.parametrize("act", ["none", "relu"])
@pytest.mark.parametrize("pat", [((1, 0), (1, 0)), ((2, 1), (3, 0)), ((4, 3), (1, 0)), ((5, 2), (2, 1))])
def test_against_brute_force(act, pat):
    rng = np.random.default_rng(7)
    B, K, N = 3, 9, 7
    (pi, oi), (po, oo) = pat
    X, W = rng.normal(size=(B, K)), rng.normal(size=(N, K))
    b, dY = rng.normal(size=N), rng.normal(size=(B, N))
    kin, kout = set(patterns.row_kept_list(K, pi, oi)), set(patterns.row_kept_list(N, po, oo))
    m_in, m_out = patterns.row_mask(K, pi, oi), patterns.row_mask(N, po, oo)
    scale = 1.0 / 0.7
    Y = fc.fc_forward(X, W, b, m_in, m_out, scale, act)
    assert np.allclose(Y, brute_forward(X.tolist(), W.tolist(), b.tolist(), kin, kout, scale, act),
                       rtol=1e-13, atol=1e-13)
    dX, dW, db = fc.fc_backward(X, W, Y, dY, m_in, m_out, scale, act)
    bX, bW, bb = brute_backward(X.tolist(), W.tolist(), Y.tolist(), dY.tolist(), kin, kout, scale, act)
    assert np.allclose(dX, bX, rtol=1e-13, atol=1e-13)
    assert np.allclose(dW, bW, rtol=1e-13, atol=1e-13)
    assert np.allclose(db, bb, rtol=1e-13, atol=1e-13)


def test_masked_equals_compacted_bitwise_all_patterns():
    rng = np.random.default_rng(11)
    B = 3
    for K, N in [(7, 5), (12, 12), (1, 3)]:
        X = rng.integers(-4, 5, size=(B, K)).astype(float)
        W = rng.integers(-4, 5, size=(N, K)).astype(float)
        b = rng.integers(-4, 5, size=N).astype(float)
        dY = rng.integers(-4, 5, size=(B, N)).astype(float)
        for (pi, oi), (po, oo) in itertools.product(
                [(d, o) for d in range(1, 6) for o in range(d)], repeat=2):
            Sin, Sout = patterns.row_kept_list(K, pi, oi), patterns.row_kept_list(N, po, oo)
            m_in, m_out = patterns.row_mask(K, pi, oi), patterns.row_mask(N, po, oo)
            for act in ("none", "relu"):
                Y = fc.fc_forward(X, W, b, m_in, m_out, 2.0, act)
                # compact: gather, multiply, scatter
                Xc, Wc = X[:, Sin], W[np.ix_(Sout, Sin)]
                Zc = Xc @ Wc.T + b[Sout]
                Ac = np.maximum(Zc, 0) if act == "relu" else Zc
                Yc = np.zeros((B, N))
                Yc[:, Sout] = 2.0 * Ac
                assert np.array_equal(Y, Yc)
                dX, dW, db = fc.fc_backward(X, W, Y, dY, m_in, m_out, 2.0, act)
                Gc = 2.0 * dY[:, Sout] * ((Y[:, Sout] > 0) if act == "relu" else 1.0)
                dXc = np.zeros((B, K))
                dXc[:, Sin] = Gc @ Wc
                dWc = np.zeros((N, K))
                dWc[np.ix_(Sout, Sin)] = Gc.T @ Xc
                dbc = np.zeros(N)
                dbc[Sout] = Gc.sum(0)
                assert np.array_equal(dX, dXc) and np.array_equal(dW, dWc) and np.array_equal(db, dbc)


@pytest.mark.parametrize("act", ["none", "relu"])
def test_backward_is_the_derivative_of_forward(act):
    rng = np.random.default_rng(3)
    B, K, N = 4, 6, 5
    X, W, b, dY = rng.normal(size=(B, K)), rng.normal(size=(N, K)), rng.normal(size=N), rng.normal(size=(B, N))
    m_in, m_out = patterns.row_mask(K, 2, 0), patterns.row_mask(N, 3, 1)
    scale = 1.7

    def L(X_, W_, b_):
        return float((fc.fc_forward(X_, W_, b_, m_in, m_out, scale, act) * dY).sum())

    Y = fc.fc_forward(X, W, b, m_in, m_out, scale, act)
    dX, dW, db = fc.fc_backward(X, W, Y, dY, m_in, m_out, scale, act)
    h = 1e-6
    for A, dA, which in ((X, dX, 0), (W, dW, 1), (b, db, 2)):
        num = np.zeros_like(A)
        for idx in np.ndindex(A.shape):
            Ap, Am = A.copy(), A.copy()
            Ap[idx] += h
            Am[idx] -= h
            args_p = [X, W, b]
            args_m = [X, W, b]
            args_p[which], args_m[which] = Ap, Am
            num[idx] = (L(*args_p) - L(*args_m)) / (2 * h)
        assert np.allclose(num, dA, rtol=1e-6, atol=1e-7)


def test_rate_zero_is_the_plain_layer():
    rng = np.random.default_rng(5)
    X, W = rng.normal(size=(2, 3)), rng.normal(size=(4, 3))
    ones_in, ones_out = patterns.row_mask(3, 1, 0), patterns.row_mask(4, 1, 0)
    Y = fc.fc_forward(X, W, None, ones_in, ones_out)
    want = [[sum(X[s][k] * W[n][k] for k in range(3)) for n in range(4)] for s in range(2)]
    assert np.allclose(Y, want, rtol=1e-14, atol=0)


def test_sgd_momentum_pinned_to_torch_sgd():
    """The restricted update equals torch.optim.SGD(momentum, no dampening) on
    the kept entries over several steps (a library routine), leaves dropped
    entries and their momentum as they were, and with nothing dropped is
    torch's update of the whole matrix."""
    import torch
    rng = np.random.default_rng(5)
    N, K, lr, mu = 7, 9, 0.01, 0.9
    for (po, oo), (pi, oi) in [((1, 0), (1, 0)), ((2, 1), (3, 0)), ((4, 3), (1, 0))]:
        m_out, m_in = patterns.row_mask(N, po, oo), patterns.row_mask(K, pi, oi)
        W0 = rng.standard_normal((N, K))
        b0 = rng.standard_normal(N)
        rows = np.flatnonzero(m_out)
        cols = np.flatnonzero(m_in)
        Wt = torch.tensor(W0[np.ix_(rows, cols)], requires_grad=True)
        bt = torch.tensor(b0[rows], requires_grad=True)
        opt = torch.optim.SGD([Wt, bt], lr=lr, momentum=mu)
        W, V, b, Vb = W0.copy(), np.zeros((N, K)), b0.copy(), np.zeros(N)
        for _ in range(3):
            dW = rng.standard_normal((N, K))
            db = rng.standard_normal(N)
            opt.zero_grad()
            Wt.grad = torch.tensor(dW[np.ix_(rows, cols)])
            bt.grad = torch.tensor(db[rows])
            opt.step()
            W, V, b, Vb = fc.sgd_momentum(W, V, dW, m_out, m_in, lr, mu, b, Vb, db)
        np.testing.assert_allclose(W[np.ix_(rows, cols)], Wt.detach().numpy(), rtol=1e-14, atol=1e-15)
        np.testing.assert_allclose(b[rows], bt.detach().numpy(), rtol=1e-14, atol=1e-15)
        dropped = np.outer(m_out, m_in) == 0
        assert np.array_equal(W[dropped], W0[dropped]) and not V[dropped].any()
        assert np.array_equal(b[m_out == 0], b0[m_out == 0]) and not Vb[m_out == 0].any()
