"""GPU parity of the LSTM layer under a tile pattern on its weights (the tile
pattern of Sec. III-B applied to the LSTM's products, Sec. IV-C) against the
fp64 oracle LSTM run on W * M, through the C ABI."""
import numpy as np
import pytest
import torch

from gpu_util import device, f64, to_dev
from oracle import lstm as olstm
from oracle import patterns as opat
from oracle import prng as oprng
from paper_1805_08939_amd import api, synth

pytestmark = pytest.mark.gpu

TOL = 1e-4  # normwise per tensor, fp32


def check(got, want, what):
    got, want = np.asarray(got, np.float64), np.asarray(want, np.float64)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    assert np.isfinite(got).all(), what
    scale = np.abs(want).max()
    err = np.abs(got - want).max() / (scale if scale > 0 else 1.0)
    assert err <= TOL, f"{what}: normwise error {err:.3e}"


def run(T, B, I, H, tile, words_of, seed, with_state=True):
    d = device()
    g = synth.generator(seed)
    X = synth.uniform(g, (T, B, I), 0.1)
    W = synth.uniform(g, (4 * H, I + H), 0.1)
    b = synth.uniform(g, (4 * H,), 0.1)
    h0 = synth.uniform(g, (B, H), 0.5) if with_state else None
    c0 = synth.uniform(g, (B, H), 0.5) if with_state else None
    dHs = synth.normal(g, (T, B, H))
    dhT = synth.normal(g, (B, H)) if with_state else None
    dcT = synth.normal(g, (B, H)) if with_state else None
    tn, tk = 4 * H // tile, (I + H) // tile
    words = words_of(tn, tk)
    M = opat.tile_mask(words, tn, tk, tile)
    Wm = f64(W) * M
    ones = np.ones(H)
    Hs64, hT64, cT64, cache = olstm.lstm_forward(f64(X), Wm, f64(b), ones, None if h0 is None else f64(h0),
                                                 None if c0 is None else f64(c0))
    dX64, dW64, db64, dh064, dc064 = olstm.lstm_backward(f64(X), Wm, ones, cache, f64(dHs),
                                                         None if dhT is None else f64(dhT),
                                                         None if dcT is None else f64(dcT))
    dW64 = dW64 * M  # the gradient with respect to W of W * M

    bits = torch.tensor(np.array(words, dtype=np.uint32).view(np.int32), device=d)
    plan_ws = torch.empty(max(api.ard_tile_plan_workspace_bytes(tn, tk), 16) // 4, dtype=torch.int32, device=d)
    nnz = opat.bitmap_popcount(words, tn * tk)
    plan = api.ard_plan_tiles(4 * H, I + H, tile, bits, nnz, plan_ws)
    desc = api.lstm_tile_desc(api.ARD_F32, T, B, I, H, plan)
    ws = torch.empty(api.ard_lstm_tile_workspace_bytes(desc) // 4 + 1, device=d)
    Xd, Wd, bd = to_dev(X.permute(0, 2, 1)), to_dev(W), to_dev(b)
    Wd_dropped = Wd.clone()
    Wd_dropped[torch.from_numpy(M == 0).to(d)] = float("nan")  # dropped tiles must never be read
    Hs = torch.full((T, H, B), 9.0, device=d)
    hT, cT = torch.full((H, B), 9.0, device=d), torch.full((H, B), 9.0, device=d)
    api.ard_lstm_tile_fwd(desc, Xd, Wd_dropped, bd, to_dev(h0.T) if h0 is not None else None,
                          to_dev(c0.T) if c0 is not None else None, Hs, hT, cT, ws)
    dX = torch.full((T, I, B), 9.0, device=d)
    dW = torch.full((4 * H, I + H), 9.0, device=d)
    db = torch.full((4 * H,), 9.0, device=d)
    dh0, dc0 = torch.full((H, B), 9.0, device=d), torch.full((H, B), 9.0, device=d)
    api.ard_lstm_tile_bwd(desc, Wd_dropped, to_dev(dHs.permute(0, 2, 1)), to_dev(dhT.T) if dhT is not None else None,
                          to_dev(dcT.T) if dcT is not None else None, ws, dX, dW, db, dh0, dc0)
    torch.cuda.synchronize()
    check(f64(Hs).transpose(0, 2, 1), Hs64, "Hs")
    check(f64(hT).T, hT64, "hT")
    check(f64(cT).T, cT64, "cT")
    check(f64(dX).transpose(0, 2, 1), dX64, "dX")
    check(f64(dW), dW64, "dW")
    check(f64(db), db64, "db")
    check(f64(dh0).T, dh064, "dh0")
    check(f64(dc0).T, dc064, "dc0")
    assert not f64(dW)[M == 0].any()


@pytest.mark.parametrize("tile", [32, 64])
@pytest.mark.parametrize("kind", ["bernoulli", "tdp", "all"])
def test_patterns(tile, kind):
    def words_of(tn, tk):
        if kind == "bernoulli":
            return oprng.tile_bitmap_bernoulli(tn, tk, 0.5, 8939, 3, 9)
        if kind == "tdp":
            return oprng.tile_bitmap_tdp(tn, tk, 3, 1)
        return oprng.tile_bitmap_tdp(tn, tk, 1, 0)
    run(4, 16, 2 * tile, tile, tile, words_of, seed=tile + len(kind))


def test_larger_layer():
    run(6, 64, 256, 192, 64, lambda tn, tk: oprng.tile_bitmap_bernoulli(tn, tk, 0.4, 8939, 1, 2), seed=11,
        with_state=False)


def test_random_shapes_and_patterns():
    """8 random layers: 32- or 64-tiles, 1-4 steps, batch 1-64, input and hidden
    sizes of 1-8 and 1-6 tiles, a Bernoulli bitmap (drop rate 0-0.9) or the
    tile pattern of a period and offset; the case is printed before it runs."""
    rng = np.random.default_rng(1805)
    for i in range(8):
        tile = int(rng.choice([32, 64]))
        T, B = int(rng.integers(1, 5)), int(rng.choice([1, 8, 16, 20, 64]))
        I, H = tile * int(rng.integers(1, 9)), tile * int(rng.integers(1, 7))
        if rng.random() < 0.5:
            p, seed = float(rng.uniform(0.0, 0.9)), int(rng.integers(1, 1000))
            words_of = lambda tn, tk, p=p, seed=seed: oprng.tile_bitmap_bernoulli(tn, tk, p, seed, 0, 0)
            what = f"bernoulli p={p:.2f}"
        else:
            q = int(rng.integers(1, 6))
            off = int(rng.integers(0, q))
            words_of = lambda tn, tk, q=q, off=off: oprng.tile_bitmap_tdp(tn, tk, q, off)
            what = f"tdp ({q}, {off})"
        state = bool(rng.random() < 0.5)
        print(f"case {i}: tile={tile} T={T} B={B} I={I} H={H} {what} state={state}", flush=True)
        run(T, B, I, H, tile, words_of, seed=40 + i, with_state=state)


def test_invalid():
    d = device()
    words = oprng.tile_bitmap_tdp(4, 3, 1, 0)
    bits = torch.tensor(np.array(words, dtype=np.uint32).view(np.int32), device=d)
    plan_ws = torch.empty(max(api.ard_tile_plan_workspace_bytes(4, 3), 16) // 4, dtype=torch.int32, device=d)
    plan = api.ard_plan_tiles(128, 96, 32, bits, 12, plan_ws)
    desc = api.lstm_tile_desc(api.ARD_F32, 2, 4, 64, 64, plan)  # the plan covers 128 x 96, W is 256 x 128
    with pytest.raises(api.ArdError):
        api.ard_lstm_tile_workspace_bytes(desc) or api.ard_lstm_tile_fwd(
            desc, torch.zeros(1, device=d), torch.zeros(1, device=d), None, None, None, torch.zeros(1, device=d),
            None, None, torch.zeros(1, device=d))
