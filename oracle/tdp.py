"""Layer under a tile-based dropout pattern (Sec. III-B), fp64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Tiles of the weight matrix are the unit dropped: with M the 0/1 element mask
of W[N][K] (the kept-tile grid expanded to tile x tile blocks) the layer is a
DropConnect-style synapse dropout with the mask applied in both passes:

    Y  = scale * X (W * M)^T
    dX = scale * dY (W * M)
    dW = scale * M * (dY^T X)

Logical layout: X [B][K], W [N][K], Y and dY [B][N].
"""

import numpy as np


def tdp_forward(X, W, M, scale=1.0):
    return scale * (np.asarray(X, np.float64) @ (np.asarray(W, np.float64) * M).T)


def tdp_backward(X, W, dY, M, scale=1.0):
    """Returns (dX, dW)."""
    X = np.asarray(X, np.float64)
    W = np.asarray(W, np.float64)
    dY = np.asarray(dY, np.float64)
    dX = scale * (dY @ (W * M))
    dW = scale * M * (dY.T @ X)
    return dX, dW
