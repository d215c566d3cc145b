"""GPU parity of the benchmark's own timed step: the MLP 784-2048-2048-10
(fp32, batch 128, ReLU) step exactly as bench.py runs it (patterns sampled
from K(p) per step, list-free plans, compact weights gathered per step, the
one-call layer backward with the ReLU gate of the layer below applied by
bwd_data, SKIP mode), checked layer by layer against the fp64 oracle fed the
same layer inputs and the same stored ReLU outputs (so that both sides take
the same gating decisions)."""
import os
import sys

import numpy as np
import pytest
import torch

from gpu_util import F32_TOL, compare, full_weight_grad
from oracle import fc as ofc
from oracle import patterns as opat
from oracle import prng as oprng

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def _host(t):
    """Feature-major device tensor -> [B][features] fp64 array."""
    return t.double().cpu().numpy().T.copy()


@pytest.fixture(scope="module")
def mlp():
    import bench
    spec = dict(bench.WORKLOADS["mlp784"])
    spec.pop("cls")
    return bench.Mlp(**spec)


@pytest.mark.parametrize("p", [0.5, 0.7, 0.0])
def test_mlp784_step_against_oracle(mlp, p):
    mlp.set_rate(p)
    # steps whose patterns differ: both hidden layers dropped, one of them
    # whole, and (at p = 0) nothing dropped
    for it in (3, 11, 27):
        pats = mlp.patterns(it)
        for l, (per, off) in enumerate(pats):
            assert (per, off) == oprng.sample_row_pattern(mlp.K, 8939, l + 1, it)
        for t in mlp.dW + mlp.db:
            t.fill_(-3.25)  # SKIP: dropped entries must keep this value
        mlp.step(it)
        torch.cuda.synchronize()
        dims, L = mlp.dims, mlp.L
        masks = [np.ones(dims[0])] + [opat.row_mask(dims[l + 1], *pats[l]) for l in range(L - 1)] + \
                [np.ones(dims[-1])]
        acts = [_host(mlp.X0)] + [_host(y) for y in mlp.Y]
        W = [mlp.full_weight(l).double().cpu().numpy() for l in range(mlp.L)]
        for l in range(L):
            act = "relu" if l < L - 1 else "none"
            m_in, m_out = masks[l], masks[l + 1]
            X = acts[l]
            want = ofc.fc_forward(X, W[l], None, m_in, m_out, 1.0, act)
            norm = (np.abs(X * m_in[None, :]) @ np.abs(W[l]).T) * m_out[None, :]
            keep = m_out > 0
            compare(acts[l + 1][:, keep], want[:, keep], norm[:, keep], F32_TOL, f"Y{l} it{it}")
            # backward: the step passes each layer its output gradient already
            # gated (by the layer above's bwd_data through Xgate, or the top's
            # linear output), so G = m_out * dY
            dYl = _host(mlp.dY[l])
            dX, dW, db = ofc.fc_backward(X, W[l], None, dYl, m_in, m_out, 1.0, "none")
            G = ofc.fc_output_grad(None, dYl, m_out, 1.0, "none")
            kw = np.outer(m_out, m_in) > 0
            got_dW = full_weight_grad(mlp, l, pats, -3.25)
            compare(got_dW[kw], dW[kw], ((np.abs(G).T @ np.abs(X)) * np.outer(m_out, m_in))[kw], F32_TOL,
                    f"dW{l} it{it}")
            assert (got_dW[~kw] == -3.25).all(), f"dW{l}: dropped entries were written"
            got_db = mlp.db[l].double().cpu().numpy()
            compare(got_db[m_out > 0], db[m_out > 0], np.abs(G).sum(0)[m_out > 0], F32_TOL, f"db{l} it{it}")
            assert (got_db[m_out == 0] == -3.25).all()
            if l > 0:
                # dY[l - 1] = dX gated by [Y_{l-1} > 0] (the layer below's ReLU)
                gate = acts[l] > 0
                got_dX = _host(mlp.dY[l - 1])
                keep_in = m_in > 0
                ndX = (np.abs(G) @ np.abs(W[l])) * m_in[None, :] * gate
                compare(got_dX[:, keep_in], (dX * gate)[:, keep_in], ndX[:, keep_in], F32_TOL, f"dX{l} it{it}")


def test_lstm_stack_step_against_oracle():
    """Two stacked LSTM layers as the benchmark's stacked workload runs them
    (each layer's hidden pattern from K(p), the upper layer's input plan the
    lower layer's pattern, BPTT from the top): every layer's outputs and
    gradients against the oracle's stack, normwise per tensor."""
    import bench
    from oracle import lstm as olstm
    st = bench.LstmStack("stack", T=4, batch=8, inputs=48, hidden=40, layers=2, dtype="f32", seed=3)
    st.set_rate(0.5)
    it = next(i for i in range(200) if all(pt[0] > 1 for pt in st.patterns(i)))
    for i in (it, 0):
        pats, _ = st.step(i)
        torch.cuda.synchronize()
        st.host_copies()
        masks = [opat.row_mask(st.H, *pt) for pt in pats]
        X = st._host["X"]
        caches = []
        for l in range(st.NL):
            m_in = masks[l - 1] if l > 0 else None
            Hs, _, _, cache = olstm.lstm_forward(X, st._host["W"][l], st._host["b"][l], masks[l], m_in=m_in)
            got = st.Hs[l].double().cpu().numpy().transpose(0, 2, 1)
            err = np.abs(got - Hs).max() / np.abs(Hs).max()
            assert err <= F32_TOL, f"Hs{l}: {err:.3e}"
            caches.append((X, cache, m_in))
            X = Hs
        dH = st._host["dHs"]
        for l in reversed(range(st.NL)):
            Xl, cache, m_in = caches[l]
            dX, dW, db, _, _ = olstm.lstm_backward(Xl, st._host["W"][l], masks[l], cache, dH, m_in=m_in)
            for name, got, want in (("dW", st.dW[l], dW), ("db", st.db[l], db)):
                g = got.double().cpu().numpy()
                err = np.abs(g - want).max() / np.abs(want).max()
                assert err <= F32_TOL, f"{name}{l}: {err:.3e}"
            if l > 0:
                g = st.dX[l].double().cpu().numpy().transpose(0, 2, 1)
                err = np.abs(g - dX).max() / np.abs(dX).max()
                assert err <= F32_TOL, f"dX{l}: {err:.3e}"
            dH = dX
