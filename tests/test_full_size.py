"""Element-by-element parity at the benchmark's full sizes, in the launch
configuration bench.py times (its own workload objects and steps), against the
fp64 oracle:

* the wide MLP 8192-8192-8192-8192 (bf16, batch 2048) under row patterns drawn
  from K(0.7): every kept entry of every layer's Y, dX, dW and db
  (Sec. III-A);
* the single FC layer 784 -> 512 (fp32, batch 64, period 2);
* the tile-pattern layer 4096 x 4096 (bf16, batch 512, 64 x 64 tiles kept by a
  device-drawn Bernoulli bitmap): every entry of Y and dX and every kept entry
  of dW (Sec. III-B);
* the LSTM with the paper's tile pattern on its weights at I = H = 1024,
  batch 64 (a shorter sequence), and the stacked 2 x 1500 LSTM at batch 20
  (Sec. IV-C), every tensor normwise.

Outputs are filled with NaN before the step, so any kept entry left unwritten
fails, and in SKIP mode every dropped entry must still hold NaN. Each layer of
a network is checked on the inputs the GPU gave it (its stored activations
and, backward, its gated output gradient), so both sides take the same ReLU
decisions. The componentwise normaliser |A| |B| of a product is computed in
fp32 (it only scales the tolerance)."""
import numpy as np
import pytest
import torch

from gpu_util import BF16_TOL, F32_TOL, compare, full_weight_grad
from oracle import fc as ofc
from oracle import lstm as olstm
from oracle import patterns as opat
from oracle import prng as oprng
from oracle import tdp as otdp

pytestmark = pytest.mark.gpu


def _host(t):
    """Feature-major device tensor -> [B][features] fp64 array."""
    return t.double().cpu().numpy().T.copy()


def _abs32(a):
    return np.abs(a).astype(np.float32)


def check_mlp_step(mlp, it, tol):
    """Runs step it of the benchmark's MLP and checks every layer against the
    oracle on the layer's own GPU inputs."""
    pats = mlp.patterns(it)
    for l, (per, off) in enumerate(pats):
        assert (per, off) == oprng.sample_row_pattern(mlp.K, 8939, l + 1, it)
    nan = float("nan")
    for t in mlp.dW + mlp.db + mlp.Y + mlp.dY[:-1]:
        t.fill_(nan)
    mlp.step(it)
    torch.cuda.synchronize()
    dims, L = mlp.dims, mlp.L
    masks = [np.ones(dims[0])] + [opat.row_mask(dims[l + 1], *pats[l]) for l in range(L - 1)] + [np.ones(dims[-1])]
    for l in range(L):
        act = "relu" if l < L - 1 else "none"
        m_in, m_out = masks[l], masks[l + 1]
        Sout = np.flatnonzero(m_out)
        keep_in = m_in > 0
        X = _host(mlp.X0) if l == 0 else _host(mlp.Y[l - 1])
        Xm = np.where(keep_in[None, :], X, 0.0)  # dropped input rows hold NaN: never read
        Wl = mlp.full_weight(l)
        W = Wl[torch.from_numpy(Sout).to(Wl.device)].double().cpu().numpy()
        ones = np.ones(len(Sout))
        # forward on the kept outputs: the oracle layer with those rows of W
        want = ofc.fc_forward(Xm, W, None, m_in, ones, 1.0, act)
        Y = _host(mlp.Y[l])
        compare(Y[:, Sout], want, _abs32(Xm) @ _abs32(W).T, tol, f"Y{l} it{it}")
        assert np.isnan(Y[:, m_out == 0]).all(), f"Y{l}: dropped rows were written"
        # backward: each layer is handed its output gradient already gated
        dYl = _host(mlp.dY[l])[:, Sout]
        dX, dW, db = ofc.fc_backward(Xm, W, None, dYl, m_in, ones, 1.0, "none")
        Ga = _abs32(dYl)
        got_dW = full_weight_grad(mlp, l, pats, nan)[Sout]
        compare(got_dW[:, keep_in], dW[:, keep_in], (Ga.T @ _abs32(Xm))[:, keep_in], tol, f"dW{l} it{it}")
        assert np.isnan(got_dW[:, ~keep_in]).all(), f"dW{l}: dropped columns were written"
        got_db = mlp.db[l].double().cpu().numpy()
        compare(got_db[Sout], db, Ga.sum(0), tol, f"db{l} it{it}")
        assert np.isnan(got_db[m_out == 0]).all()
        if l > 0:  # dY[l - 1] = dX gated by the layer below's ReLU output [Y_{l-1} > 0]
            gate = X > 0
            got_dX = _host(mlp.dY[l - 1])
            compare(got_dX[:, keep_in], (dX * gate)[:, keep_in], ((Ga @ _abs32(W)) * gate)[:, keep_in], tol,
                    f"dX{l} it{it}")
            assert np.isnan(got_dX[:, ~keep_in]).all(), f"dX{l}: dropped rows were written"
    return pats


@pytest.fixture(scope="module")
def wide_mlp():
    import bench
    spec = dict(bench.WORKLOADS["mlp8192"])
    spec.pop("cls")
    return bench.Mlp(**spec)


def test_wide_mlp_step_full_size(wide_mlp):
    """Steps of the wide MLP at p = 0.7: one with both hidden layers dropped
    at large periods (the narrowest kept sets), one with the first hidden
    layer whole and the second dropped."""
    mlp = wide_mlp
    mlp.set_rate(0.7)
    its = [next(i for i in range(1000) if min(pt[0] for pt in mlp.patterns(i)) >= 11),
           next(i for i in range(1000) if mlp.patterns(i)[0][0] == 16),
           next(i for i in range(1000) if mlp.patterns(i)[0][0] == 1 and mlp.patterns(i)[1][0] > 1)]
    for it in its:
        check_mlp_step(mlp, it, BF16_TOL)


def test_single_fc_layer_step_full_size():
    import bench
    spec = dict(bench.WORKLOADS["fc784"])
    spec.pop("cls")
    fc = bench.FcLayer(**spec)
    fc.set_rate(0.5)
    fc.host_copies()
    for it in (0, 1, 7):
        nan = float("nan")
        for t in (fc.Yt, fc.dXt, fc.dW, fc.db):
            t.fill_(nan)
        pats, _ = fc.step(it)
        torch.cuda.synchronize()
        assert pats[0][0] == 2
        X, W, dY = fc._host
        m_in, m_out = np.ones(fc.K), opat.row_mask(fc.N, *pats[0])
        keep = m_out > 0
        Y64 = ofc.fc_forward(X, W, None, m_in, m_out)
        dX64, dW64, db64 = ofc.fc_backward(X, W, Y64, dY, m_in, m_out)
        G = np.abs(dY) * m_out[None, :]
        Y = _host(fc.Yt)
        compare(Y[:, keep], Y64[:, keep], (np.abs(X) @ np.abs(W).T)[:, keep], F32_TOL, "Y")
        assert np.isnan(Y[:, ~keep]).all()
        compare(_host(fc.dXt), dX64, G @ np.abs(W), F32_TOL, "dX")
        dW = fc.dW.double().cpu().numpy()
        compare(dW[keep], dW64[keep], (G.T @ np.abs(X))[keep], F32_TOL, "dW")
        assert np.isnan(dW[~keep]).all()
        db = fc.db.double().cpu().numpy()
        compare(db[keep], db64[keep], G.sum(0)[keep], F32_TOL, "db")


def test_tile_layer_full_size():
    """The benchmark's tile-pattern layer step (bitmap drawn and planned on the
    device, SKIP mode): every entry of Y and dX, every kept tile of dW."""
    import bench
    spec = dict(bench.WORKLOADS["tile4096"])
    spec.pop("cls")
    tl = bench.TileLayer(**spec)
    tl.host_copies()
    X, W, dY = tl._host
    # steps 3 and 4 in a row: step 4 runs on the plan built during step 3
    for p, it in ((0.5, 3), (0.5, 4), (0.7, 9)):
        if p != getattr(tl, "p", None):
            tl.set_rate(p)
        nan = float("nan")
        for t in (tl.Yt, tl.dXt, tl.dW):
            t.fill_(nan)
        tl.step(it)
        torch.cuda.synchronize()
        words = oprng.tile_bitmap_bernoulli(tl.tn, tl.tk, p, 8939, 0, it)
        bits = tl.bits_bufs[it % 2]  # the step's plan buffer
        assert [int(w) for w in bits.cpu().numpy().view(np.uint32)] == [int(w) for w in words]
        M = opat.tile_mask(words, tl.tn, tl.tk, tl.tile)
        Y64 = otdp.tdp_forward(X, W, M)
        dX64, dW64 = otdp.tdp_backward(X, W, dY, M)
        Wa = _abs32(W) * M.astype(np.float32)
        compare(_host(tl.Yt), Y64, _abs32(X) @ Wa.T, BF16_TOL, f"Y p{p}")
        compare(_host(tl.dXt), dX64, _abs32(dY) @ Wa, BF16_TOL, f"dX p{p}")
        dW = tl.dW.double().cpu().numpy()
        kept = M > 0
        compare(dW[kept], dW64[kept], (_abs32(dY).T @ _abs32(X))[kept], BF16_TOL, f"dW p{p}")
        assert np.isnan(dW[~kept]).all(), "dropped tiles of dW were written"


def _normwise(got, want, what, tol=F32_TOL):
    got, want = np.asarray(got, np.float64), np.asarray(want, np.float64)
    assert np.isfinite(got).all(), what
    err = np.abs(got - want).max() / np.abs(want).max()
    assert err <= tol, f"{what}: normwise error {err:.3e}"


def test_tile_lstm_full_width():
    """The tile-pattern LSTM at the benchmark's layer size (I = H = 1024,
    batch 64, 64 x 64 tiles; 3 steps instead of 35), the paper's tile pattern
    (dp, offset) from K(0.5): its per-step products split the kept-tile lists
    over fewer workgroups than the small test shapes do."""
    import bench
    lt = bench.LstmTile("lstm-tile-t3", T=3, batch=64, inputs=1024, hidden=1024, tile=64, dtype="f32", seed=1808)
    lt.set_rate(0.5)
    it = next(i for i in range(1000) if lt.patterns(i)[0][0] in (3, 5))
    nan = float("nan")
    for t in (lt.Hs, lt.dX, lt.dW, lt.db):
        t.fill_(nan)
    pats, _ = lt.step(it)
    torch.cuda.synchronize()
    X = lt.X.double().cpu().numpy().transpose(0, 2, 1)
    W, b = lt.W.double().cpu().numpy(), lt.b.double().cpu().numpy()
    dHs = lt.dHs.double().cpu().numpy().transpose(0, 2, 1)
    words = oprng.tile_bitmap_tdp(lt.tn, lt.tk, *pats[0])
    M = opat.tile_mask(words, lt.tn, lt.tk, lt.tile)
    ones = np.ones(lt.H)
    Hs, _, _, cache = olstm.lstm_forward(X, W * M, b, ones)
    dX, dW, db, _, _ = olstm.lstm_backward(X, W * M, ones, cache, dHs)
    _normwise(lt.Hs.double().cpu().numpy().transpose(0, 2, 1), Hs, "Hs")
    _normwise(lt.dX.double().cpu().numpy().transpose(0, 2, 1), dX, "dX")
    got_dW = lt.dW.double().cpu().numpy()
    _normwise(got_dW, dW * M, "dW")
    assert not got_dW[M == 0].any()
    _normwise(lt.db.double().cpu().numpy(), db, "db")


def test_stacked_lstm_full_width():
    """The stacked 2 x 1500 LSTM at batch 20 (3 steps instead of 35), each
    layer's hidden pattern from K(0.5), the upper layer's input plan the lower
    layer's pattern: every layer's Hs, dW, db and the upper layer's dX."""
    import bench
    st = bench.LstmStack("stack-t3", T=3, batch=20, inputs=1500, hidden=1500, layers=2, dtype="f32", seed=1810)
    st.set_rate(0.5)
    it = next(i for i in range(1000) if all(pt[0] > 1 for pt in st.patterns(i)))
    pats, _ = st.step(it)
    torch.cuda.synchronize()
    st.host_copies()
    masks = [opat.row_mask(st.H, *pt) for pt in pats]
    X = st._host["X"]
    caches = []
    for l in range(st.NL):
        m_in = masks[l - 1] if l > 0 else None
        Hs, _, _, cache = olstm.lstm_forward(X, st._host["W"][l], st._host["b"][l], masks[l], m_in=m_in)
        _normwise(st.Hs[l].double().cpu().numpy().transpose(0, 2, 1), Hs, f"Hs{l}")
        caches.append((X, cache, m_in))
        X = Hs
    dH = st._host["dHs"]
    for l in reversed(range(st.NL)):
        Xl, cache, m_in = caches[l]
        dX, dW, db, _, _ = olstm.lstm_backward(Xl, st._host["W"][l], masks[l], cache, dH, m_in=m_in)
        _normwise(st.dW[l].double().cpu().numpy(), dW, f"dW{l}")
        _normwise(st.db[l].double().cpu().numpy(), db, f"db{l}")
        if l > 0:
            _normwise(st.dX[l].double().cpu().numpy().transpose(0, 2, 1), dX, f"dX{l}")
        dH = dX


@pytest.mark.parametrize("period", [3, 8])
def test_lstm_full_width_small_kept_sets(period):
    """The 1024/1024 LSTM at batch 64 (4 steps instead of 35) with hidden
    period 3 (342 kept units) and 8 (128): the kept sets whose backward steps
    run the fused one-kernel recurrence and whose forward steps run on 16 x 16
    tiles. Hs, hT, cT, dX, dW, db, dh0 and dc0 against the oracle."""
    import bench
    wl = bench.Lstm("lstm-t4", T=4, batch=64, inputs=1024, hidden=1024, dtype="f32", seed=1811)
    api = wl.api
    api.ard_plan_rows(wl.H, period, 1, wl.idx, wl.stream, plan=wl.plan)
    d = wl.desc
    api.ard_lstm_fwd(d, wl.X, wl.W, wl.b, None, None, wl.Hs, wl.hT, wl.cT, wl.ws, wl.stream)
    api.ard_lstm_bwd(d, wl.X, wl.dHs, None, None, wl.ws, wl.dX, wl.dW, wl.db, wl.dh0, wl.dc0, wl.stream)
    torch.cuda.synchronize()
    wl.host_copies()
    X, W, b, dHs = wl._host
    m = opat.row_mask(wl.H, period, 1)
    Hs, hT, cT, cache = olstm.lstm_forward(X, W, b, m)
    dX, dW, db, dh0, dc0 = olstm.lstm_backward(X, W, m, cache, dHs)
    t = lambda a: a.double().cpu().numpy()
    _normwise(t(wl.Hs).transpose(0, 2, 1), Hs, "Hs")
    _normwise(t(wl.hT).T, hT, "hT")
    _normwise(t(wl.cT).T, cT, "cT")
    _normwise(t(wl.dX).transpose(0, 2, 1), dX, "dX")
    _normwise(t(wl.dW), dW, "dW")
    _normwise(t(wl.db), db, "db")
    _normwise(t(wl.dh0).T, dh0, "dh0")
    _normwise(t(wl.dc0).T, dc0, "dc0")
