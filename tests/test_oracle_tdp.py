"""Pins of the oracle's tile-pattern layer (Sec. III-B)."""
import numpy as np
import pytest

from oracle import patterns, prng, tdp


def test_against_brute_force_and_compaction():
    rng = np.random.default_rng(2)
    tile, tn, tk, B = 2, 3, 4, 3
    N, K = tn * tile, tk * tile
    X = rng.integers(-3, 4, size=(B, K)).astype(float)
    W = rng.integers(-3, 4, size=(N, K)).astype(float)
    dY = rng.integers(-3, 4, size=(B, N)).astype(float)
    for words in (prng.tile_bitmap_tdp(tn, tk, 3, 1), prng.tile_bitmap_bernoulli(tn, tk, 0.5, 4, 0, 1),
                  prng.tile_bitmap_tdp(tn, tk, 1, 0)):
        M = patterns.tile_mask(words, tn, tk, tile)
        grid = patterns.bitmap_to_grid(words, tn, tk)
        Y = tdp.tdp_forward(X, W, M, 1.5)
        dX, dW = tdp.tdp_backward(X, W, dY, M, 1.5)
        # brute force over kept tiles only (the compacted tile computation)
        Yb = np.zeros((B, N))
        dXb = np.zeros((B, K))
        dWb = np.zeros((N, K))
        for a in range(tn):
            for c in range(tk):
                if not grid[a, c]:
                    continue
                rs, cs = slice(a * tile, (a + 1) * tile), slice(c * tile, (c + 1) * tile)
                Yb[:, rs] += 1.5 * X[:, cs] @ W[rs, cs].T
                dXb[:, cs] += 1.5 * dY[:, rs] @ W[rs, cs]
                dWb[rs, cs] = 1.5 * dY[:, rs].T @ X[:, cs]
        assert np.array_equal(Y, Yb) and np.array_equal(dX, dXb) and np.array_equal(dW, dWb)


def test_all_kept_is_dense_and_all_dropped_is_zero():
    rng = np.random.default_rng(9)
    X, W = rng.normal(size=(3, 8)), rng.normal(size=(4, 8))
    ones = patterns.tile_mask(prng.tile_bitmap_bernoulli(2, 4, 0.0, 0, 0, 0), 2, 4, 2)
    want = [[sum(X[s][k] * W[n][k] for k in range(8)) for n in range(4)] for s in range(3)]
    assert np.allclose(tdp.tdp_forward(X, W, ones), want, rtol=1e-14)
    zeros = patterns.tile_mask(prng.tile_bitmap_bernoulli(2, 4, 1.0, 0, 0, 0), 2, 4, 2)
    assert not tdp.tdp_forward(X, W, zeros).any()


def test_backward_is_the_derivative_of_forward():
    rng = np.random.default_rng(4)
    X, W, dY = rng.normal(size=(3, 6)), rng.normal(size=(4, 6)), rng.normal(size=(3, 4))
    M = patterns.tile_mask(prng.tile_bitmap_tdp(2, 3, 2, 0), 2, 3, 2)
    dX, dW = tdp.tdp_backward(X, W, dY, M, 0.5)
    h = 1e-6
    for A, dA, is_x in ((X, dX, True), (W, dW, False)):
        num = np.zeros_like(A)
        for idx in np.ndindex(A.shape):
            Ap, Am = A.copy(), A.copy()
            Ap[idx] += h
            Am[idx] -= h
            fp = tdp.tdp_forward(Ap, W, M, 0.5) if is_x else tdp.tdp_forward(X, Ap, M, 0.5)
            fm = tdp.tdp_forward(Am, W, M, 0.5) if is_x else tdp.tdp_forward(X, Am, M, 0.5)
            num[idx] = ((fp - fm) * dY).sum() / (2 * h)
        assert np.allclose(num, dA, rtol=1e-6, atol=1e-8)
