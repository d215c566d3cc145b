"""GPU parity of the LSTM layer with hidden-unit row dropout (Sec. IV-C)."""
import numpy as np
import pytest
import torch

from gpu_util import device, f64, row_plan, to_dev
from oracle import lstm as olstm
from oracle import patterns as opat
from oracle import prng as oprng
from paper_1805_08939_amd import api, synth

pytestmark = pytest.mark.gpu

TOL = 1e-4  # normwise per tensor, fp32


def check(got, want, what, tol=TOL):
    got, want = np.asarray(got, np.float64), np.asarray(want, np.float64)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    assert np.isfinite(got).all(), what
    scale = np.abs(want).max()
    err = np.abs(got - want).max() / (scale if scale > 0 else 1.0)
    assert err <= tol, f"{what}: normwise error {err:.3e}"
    return err


def run_lstm(T, B, I, H, pattern, seed, with_state=True, with_final_grads=True, a=0.1, in_pattern=(1, 0)):
    g = synth.generator(seed)
    X = synth.uniform(g, (T, B, I), a)
    W = synth.uniform(g, (4 * H, I + H), a)
    b = synth.uniform(g, (4 * H,), a)
    h0 = synth.uniform(g, (B, H), 0.5) if with_state else None
    c0 = synth.uniform(g, (B, H), 0.5) if with_state else None
    dHs = synth.normal(g, (T, B, H))
    dhT = synth.normal(g, (B, H)) if with_final_grads else None
    dcT = synth.normal(g, (B, H)) if with_final_grads else None
    m = opat.row_mask(H, *pattern)
    m_in = opat.row_mask(I, *in_pattern)
    Hs64, hT64, cT64, cache = olstm.lstm_forward(f64(X), f64(W), f64(b), m,
                                                 None if h0 is None else f64(h0), None if c0 is None else f64(c0),
                                                 m_in=m_in)
    dX64, dW64, db64, dh064, dc064 = olstm.lstm_backward(
        f64(X), f64(W), m, cache, f64(dHs), None if dhT is None else f64(dhT), None if dcT is None else f64(dcT),
        m_in=m_in)

    plan = None if pattern == (1, 0) else row_plan(H, *pattern)
    in_plan = None if in_pattern == (1, 0) else row_plan(I, *in_pattern, with_list=False)
    desc = api.lstm_desc(api.ARD_F32, T, B, I, H, plan, in_plan)
    ws = torch.empty(api.ard_lstm_workspace_bytes(desc) // 4 + 1, dtype=torch.float32, device=device())
    Xd = to_dev(X.permute(0, 2, 1))      # [T][I][B]
    if in_plan is not None:  # dropped inputs must never be read
        Xd[:, torch.from_numpy(m_in == 0).to(device())] = float("nan")
    Wd, bd = to_dev(W), to_dev(b)
    h0d = to_dev(h0.T) if h0 is not None else None
    c0d = to_dev(c0.T) if c0 is not None else None
    Hs = torch.full((T, H, B), 9.0, device=device())
    hT = torch.full((H, B), 9.0, device=device())
    cT = torch.full((H, B), 9.0, device=device())
    api.ard_lstm_fwd(desc, Xd, Wd, bd, h0d, c0d, Hs, hT, cT, ws)
    dHsd = to_dev(dHs.permute(0, 2, 1))
    dhTd = to_dev(dhT.T) if dhT is not None else None
    dcTd = to_dev(dcT.T) if dcT is not None else None
    dX = torch.full((T, I, B), 9.0, device=device())
    dW = torch.full((4 * H, I + H), 9.0, device=device())
    db = torch.full((4 * H,), 9.0, device=device())
    dh0 = torch.full((H, B), 9.0, device=device())
    dc0 = torch.full((H, B), 9.0, device=device())
    api.ard_lstm_bwd(desc, Xd, dHsd, dhTd, dcTd, ws, dX, dW, db, dh0, dc0)
    torch.cuda.synchronize()
    check(f64(Hs).transpose(0, 2, 1), Hs64, "Hs")
    check(f64(hT).T, hT64, "hT")
    check(f64(cT).T, cT64, "cT")
    check(f64(dX).transpose(0, 2, 1), dX64, "dX")
    check(f64(dW), dW64, "dW")
    check(f64(db), db64, "db")
    check(f64(dh0).T, dh064, "dh0")
    check(f64(dc0).T, dc064, "dc0")
    dropped = m == 0
    assert not f64(Hs)[:, dropped].any() and not f64(dW)[np.tile(dropped, 4)].any()
    return Hs


@pytest.mark.parametrize("shape,pattern,in_pattern", [
    ((3, 5, 6, 10), (2, 1), (3, 1)),         # unaligned: the register-staged paths
    ((2, 8, 12, 10), (3, 0), (2, 1)),
    ((2, 8, 12, 10), (1, 0), (4, 3)),
    ((4, 64, 96, 200), (2, 1), (3, 2)),      # aligned: the direct-load GEMMs and step kernels
    ((8, 64, 512, 384), (2, 0), (2, 1)),
])
def test_input_pattern(shape, pattern, in_pattern):
    """Stacked layers: the input rows dropped by the layer below are skipped
    (the input products and the input columns of W shrink with them)."""
    run_lstm(*shape, pattern, seed=sum(shape), in_pattern=in_pattern)


@pytest.mark.parametrize("pattern", [(1, 0), (2, 1), (3, 0), (7, 6), (16, 12)])
def test_tiny_patterns(pattern):
    run_lstm(3, 5, 6, 10, pattern, seed=sum(pattern))
    run_lstm(2, 4, 8, 10, pattern, seed=7, with_state=False, with_final_grads=False)


@pytest.mark.parametrize("shape,pattern", [((4, 40, 68, 100), (3, 1)), ((3, 37, 33, 70), (2, 0)),
                                           ((5, 96, 128, 160), (4, 3)), ((1, 8, 12, 64), (5, 2)),
                                           # split forward recurrence on unaligned operands (KW = 370)
                                           ((3, 36, 70, 600), (2, 1))])
def test_multi_tile_and_unaligned(shape, pattern):
    T, B, I, H = shape
    run_lstm(T, B, I, H, pattern, seed=B)


@pytest.mark.parametrize("shape", [(3, 64, 256, 1024), (2, 48, 128, 2048)])
def test_all_units_kept_wide_recurrence_tiles(shape):
    """1024 and 2048 kept units at batch 64 and 48: the backward recurrence on
    32 x 64 tiles (one tile column holds the batch)."""
    run_lstm(*shape, (1, 0), seed=sum(shape), with_state=True)


@pytest.mark.parametrize("shape,pattern,in_pattern", [((35, 20, 640, 320), (2, 1), (1, 0)),
                                                      ((35, 20, 768, 320), (2, 0), (2, 1))])
def test_small_batch_steps_on_narrow_tiles(shape, pattern, in_pattern):
    """Batch 20 over 35 steps: the step-batched input projection (and, with
    every input kept, the input gradient) has 20 columns per step and at
    least 160 row tiles of 128, so it runs on 128 x 32 tiles."""
    run_lstm(*shape, pattern, seed=sum(shape), in_pattern=in_pattern)


def random_lstm_cases(n, seed):
    """n seeded layer shapes: 1-5 steps, batch 1-100, input and hidden sizes
    1-700, a hidden pattern of period 1-16 and (in a third of the cases) an
    input pattern, each keeping at least one unit; initial state and final
    gradients present or absent."""
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        T = int(rng.integers(1, 6))
        B = int(rng.choice([1, 2, 5, 8, 16, 20, 33, 64, 100]))
        I, H = int(rng.integers(1, 701)), int(rng.integers(1, 701))
        q = 1 if rng.random() < 0.25 else int(rng.integers(2, 17))
        pat = (q, int(rng.integers(0, q)))
        qi = int(rng.integers(2, 9)) if rng.random() < 0.33 else 1
        ipat = (qi, int(rng.integers(0, qi)))
        if opat.row_kept_count(H, *pat) < 1 or opat.row_kept_count(I, *ipat) < 1:
            continue
        out.append((T, B, I, H, pat, ipat, bool(rng.random() < 0.5), bool(rng.random() < 0.5)))
    return out


def test_random_shapes_and_patterns():
    """Forward and backward of 10 random layers (see random_lstm_cases) against
    the oracle; the case is printed before it runs."""
    for i, (T, B, I, H, pat, ipat, state, finals) in enumerate(random_lstm_cases(10, 1805)):
        print(f"case {i}: T={T} B={B} I={I} H={H} pattern={pat} input={ipat} state={state} finals={finals}",
              flush=True)
        run_lstm(T, B, I, H, pat, seed=100 + i, with_state=state, with_final_grads=finals, in_pattern=ipat)


def test_full_config_lstm_1024():
    """Single LSTM layer fp32, input 1024, hidden 1024, 35 steps, batch 64, hidden
    units dropped with period 2 (seeded offset), inputs ~ U(-0.1, 0.1)."""
    K2 = np.zeros(16)
    K2[1] = 1.0
    per, off = oprng.sample_row_pattern(K2, 8939, 0, 0)
    run_lstm(35, 64, 1024, 1024, (per, off), seed=1805 + 3, with_state=False, with_final_grads=False)


def test_bwd_on_workspace_of_another_plan():
    """A backward call whose workspace holds the forward state of another plan
    (other kept count, so another workspace layout) gives undefined gradients
    but writes only inside its outputs; the matching forward and backward run
    afterwards on the same workspace agree exactly with a fresh workspace."""
    T, B, I, H = 3, 64, 48, 96
    g = synth.generator(11)
    X = to_dev(synth.uniform(g, (T, I, B), 0.1))
    W, b = to_dev(synth.uniform(g, (4 * H, I + H), 0.1)), to_dev(synth.uniform(g, (4 * H,), 0.1))
    dHs = to_dev(synth.normal(g, (T, H, B)))
    da = api.lstm_desc(api.ARD_F32, T, B, I, H, row_plan(H, 2, 1))
    db_ = api.lstm_desc(api.ARD_F32, T, B, I, H, row_plan(H, 3, 0))
    n = max(api.ard_lstm_workspace_bytes(da), api.ard_lstm_workspace_bytes(db_)) // 4 + 1

    def outs():
        return [torch.full(sh, 9.0, device=device()) for sh in ((T, H, B), (T, I, B), (4 * H, I + H), (4 * H,))]

    # guard words after each output catch a write past its end
    guard = torch.full((4 * H * (I + H) + 4096,), 7.0, device=device())
    dW_g = guard[:4 * H * (I + H)].view(4 * H, I + H)
    ws = torch.zeros(n, device=device())
    Hs, dX, _, dbias = outs()
    api.ard_lstm_fwd(db_, X, W, b, None, None, Hs, None, None, ws)
    api.ard_lstm_bwd(da, X, dHs, None, None, ws, dX, dW_g, dbias, None, None)
    torch.cuda.synchronize()
    assert (guard[4 * H * (I + H):] == 7.0).all()
    res = []
    for w in (ws, torch.zeros(n, device=device())):
        Hs, dX, dW, dbias = outs()
        api.ard_lstm_fwd(da, X, W, b, None, None, Hs, None, None, w)
        api.ard_lstm_bwd(da, X, dHs, None, None, w, dX, dW, dbias, None, None)
        res.append((Hs, dX, dW, dbias))
    torch.cuda.synchronize()
    for x, y in zip(*res):
        assert torch.equal(x, y)


def test_deterministic():
    a = run_lstm(4, 64, 64, 96, (2, 1), seed=5)
    b = run_lstm(4, 64, 64, 96, (2, 1), seed=5)
    assert torch.equal(a, b)


def test_invalid():
    d = device()
    desc = api.lstm_desc(api.ARD_BF16, 2, 4, 8, 8)
    with pytest.raises(api.ArdError):
        api.ard_lstm_fwd(desc, torch.zeros(1, device=d), torch.zeros(1, device=d), None, None, None,
                         torch.zeros(1, device=d), None, None, torch.zeros(1, device=d))
    desc = api.lstm_desc(api.ARD_F32, 2, 4, 8, 8)
    small = torch.zeros(4, device=d)
    with pytest.raises(api.ArdError) as e:
        api.ard_lstm_fwd(desc, torch.zeros(64, device=d), torch.zeros(512, device=d), None, None, None,
                         torch.zeros(64, device=d), None, None, small)
    assert e.value.status == 5
    # the LSTM reads the kept-unit list: a list-free plan that drops units is rejected
    plan = api.ard_plan_rows(8, 2, 1, None)
    desc = api.lstm_desc(api.ARD_F32, 2, 4, 8, 8, plan)
    with pytest.raises(api.ArdError) as e:
        api.ard_lstm_fwd(desc, torch.zeros(64, device=d), torch.zeros(512, device=d), None, None, None,
                         torch.zeros(64, device=d), None, None, torch.zeros(1 << 20, device=d))
    assert e.value.status == api.ARD_ERR_INVALID_ARG and "d_idx" in e.value.message
