"""GPU parity of the FC layer under row patterns (fwd / bwd_data / bwd_weight)
against the fp64 oracle, through the C ABI."""
import itertools

import numpy as np
import pytest
import torch

from gpu_util import ard_dtype, compare, device, f64, row_plan, to_dev, tol, workspace
from oracle import fc as ofc
from oracle import patterns as opat
from oracle import prng as oprng
from paper_1805_08939_amd import api, synth

pytestmark = pytest.mark.gpu

ACTS = {"none": api.ARD_ACT_NONE, "relu": api.ARD_ACT_RELU}
F32_TOL_UPD = 1e-6  # fp32 momentum and bias: a few roundings of one multiply-add


def make_inputs(dtype, B, K, N, seed, w_std=0.05, bias=True):
    g = synth.generator(seed)
    X = synth.to_storage(synth.normal(g, (B, K)), dtype)
    W = synth.to_storage(synth.normal(g, (N, K), w_std), dtype)
    b = synth.normal(g, (N,), 0.1) if bias else None
    dY = synth.to_storage(synth.normal(g, (B, N)), dtype)
    return X, W, b, dY


def run_layer(dtype, X, W, b, dY, pin, pout, act, scale, dropped, use_null_plans=True,
              sentinel=None, poison=False, lists=True):
    """Runs fwd, bwd_data and bwd_weight on the GPU and checks each against the
    oracle. Returns the GPU outputs. lists=False: list-free row plans (the FC
    calls read patterns as strided views)."""
    B, K = X.shape
    N = W.shape[0]
    m_in, m_out = opat.row_mask(K, *pin), opat.row_mask(N, *pout)
    b64 = f64(b) if b is not None else None
    Y64 = ofc.fc_forward(f64(X), f64(W), b64, m_in, m_out, scale, act)
    # the stored forward output feeds both sides' ReLU gate
    Ys = synth.to_storage(torch.from_numpy(Y64).float(), dtype)
    dX64, dW64, db64 = ofc.fc_backward(f64(X), f64(W), f64(Ys), f64(dY), m_in, m_out, scale, act)

    in_plan = None if (use_null_plans and pin == (1, 0)) else row_plan(K, *pin, with_list=lists)
    out_plan = None if (use_null_plans and pout == (1, 0)) else row_plan(N, *pout, with_list=lists)
    desc = api.fc_desc(ard_dtype(dtype), B, K, N, in_plan, out_plan, scale, ACTS[act], dropped)

    Xt, Wd, dYt, Yst = to_dev(X.T), to_dev(W), to_dev(dY.T), to_dev(Ys.T)
    if poison:  # dropped data must never enter the arithmetic
        Xt[torch.from_numpy(m_in == 0).to(device())] = float("nan")
        Wd[torch.from_numpy(m_out == 0).to(device())] = float("nan")
        Wd[:, torch.from_numpy(m_in == 0).to(device())] = float("nan")
        dYt[torch.from_numpy(m_out == 0).to(device())] = float("nan")
        Yst[torch.from_numpy(m_out == 0).to(device())] = float("nan")
    bd = to_dev(b) if b is not None else None
    sdt = synth.storage_dtype(dtype)
    fill = 0.0 if sentinel is None else sentinel
    Yt = torch.full((N, B), fill, dtype=sdt, device=device())
    dXt = torch.full((K, B), fill, dtype=sdt, device=device())
    dW = torch.full((N, K), fill, dtype=torch.float32, device=device())
    db = torch.full((N,), fill, dtype=torch.float32, device=device())

    ws = workspace(api.ard_fc_workspace_bytes(desc))
    api.ard_fc_fwd(desc, Xt, Wd, bd, Yt, ws)
    api.ard_fc_bwd_data(desc, dYt, Yst, Wd, dXt, ws)
    api.ard_fc_bwd_weight(desc, Xt, dYt, Yst, dW, db, ws)
    # the layer backward in one call (one launch where both products are
    # small): bitwise the separate calls' results
    dXt2, dW2, db2 = (torch.full_like(t, fill) for t in (dXt, dW, db))
    api.ard_fc_bwd(desc, Xt, dYt, Yst, Wd, dXt2, dW2, db2, ws)
    torch.cuda.synchronize()
    assert torch.equal(dXt2, dXt) and torch.equal(dW2, dW) and torch.equal(db2, db)
    # Y and dX of the compact layouts, checked against the oracle below: equal
    # to the full layout's up to the rounding order (a full-layout view that the
    # direct-load kernels cannot read takes the general kernel)
    alt = {"Y": [], "dX": []}
    if pin != (1, 0) and not poison:
        # the same layer with the caller compacting W once (with a gathered
        # input side the full layout compacts W itself: bitwise identical)
        cdesc = api.fc_desc(ard_dtype(dtype), B, K, N, in_plan, out_plan, scale, ACTS[act], dropped,
                            api.ARD_WEIGHTS_COMPACT)
        Wc = torch.empty(max(api.ard_fc_compact_bytes(cdesc), 16) // 2, dtype=torch.int16, device=device())
        api.ard_fc_compact_weights(cdesc, Wd, Wc)
        cws = workspace(api.ard_fc_workspace_bytes(cdesc))
        Yt2, dXt2 = Yt.clone(), dXt.clone()
        api.ard_fc_fwd(cdesc, Xt, Wc, bd, Yt2, cws)
        api.ard_fc_bwd_data(cdesc, dYt, Yst, Wc, dXt2, cws)
        torch.cuda.synchronize()
        assert torch.equal(Yt2, Yt) and torch.equal(dXt2, dXt)
        alt["Y"].append(Yt2)
        alt["dX"].append(dXt2)
    if not poison:
        # the compact weight gradient: dWc[i][j] = dW[S_out(i)][S_in(j)] bit
        # for bit, through bwd_weight and through the one-call backward
        gdesc = api.fc_desc(ard_dtype(dtype), B, K, N, in_plan, out_plan, scale, ACTS[act], dropped,
                            api.ARD_WEIGHTS_COMPACT_GRAD)
        Sin, Sout = opat.row_kept_list(K, *pin), opat.row_kept_list(N, *pout)
        ldc = api.ard_fc_compact_ld(gdesc)
        Wc = torch.empty(max(api.ard_fc_compact_bytes(gdesc), 16) // 2, dtype=torch.int16, device=device())
        api.ard_fc_compact_weights(gdesc, Wd, Wc)
        gws = workspace(api.ard_fc_workspace_bytes(gdesc))
        nc = len(Sout) * ldc
        dWc_buf = torch.full((max(nc, 4),), 7.0, device=device())  # never a null pointer
        dWc2_buf, db3, dXt3 = dWc_buf.clone(), torch.full_like(db, fill), torch.full_like(dXt, fill)
        db4, dXt4 = torch.full_like(db, fill), torch.full_like(dXt, fill)
        api.ard_fc_bwd_weight(gdesc, Xt, dYt, Yst, dWc_buf, db3, gws)
        api.ard_fc_bwd(gdesc, Xt, dYt, Yst, Wc, dXt3, dWc2_buf, db4, gws)
        api.ard_fc_bwd_data(gdesc, dYt, Yst, Wc, dXt4, gws)
        torch.cuda.synchronize()
        dWc, dWc2 = dWc_buf[:nc].view(len(Sout), ldc), dWc2_buf[:nc].view(len(Sout), ldc)
        want_c = dW[torch.tensor(Sout, dtype=torch.long, device=device())][:, torch.tensor(Sin, dtype=torch.long,
                                                                                              device=device())]
        assert torch.equal(dWc[:, :len(Sin)], want_c) and torch.equal(dWc2_buf, dWc_buf)
        assert (dWc[:, len(Sin):] == 7.0).all(), "padding columns were written"
        assert torch.equal(db3, db) and torch.equal(db4, db) and torch.equal(dXt3, dXt4)
        alt["dX"].append(dXt3)

    Xa, Wa = np.abs(f64(X) * m_in[None, :]), np.abs(f64(W))
    G = ofc.fc_output_grad(f64(Ys), f64(dY), m_out, scale, act)
    nY = abs(scale) * (Xa @ Wa.T + (np.abs(b64)[None, :] if b64 is not None else 0.0)) * m_out[None, :]
    ndX = (np.abs(G) @ Wa) * m_in[None, :]
    ndW = (np.abs(G).T @ Xa) * np.outer(m_out, m_in)
    ndb = np.abs(G).sum(0)
    t = tol(dtype)
    got = {"Y": f64(Yt).T, "dX": f64(dXt).T, "dW": f64(dW), "db": f64(db)}
    keep = {"Y": np.broadcast_to(m_out[None, :] > 0, Y64.shape),
            "dX": np.broadcast_to(m_in[None, :] > 0, dX64.shape),
            "dW": np.outer(m_out, m_in) > 0, "db": m_out > 0}
    want = {"Y": Y64, "dX": dX64, "dW": dW64, "db": db64}
    norm = {"Y": nY, "dX": ndX, "dW": ndW, "db": ndb}
    checks = [(k, v) for k, v in got.items()] + [(k, f64(v).T) for k, vs in alt.items() for v in vs]
    for k, v in checks:
        if dropped == api.ARD_DROPPED_SKIP:
            # untouched: bit-identical sentinel outside the kept sets
            assert (v[~keep[k]] == fill).all(), f"{k}: dropped entries were written"
            compare(v[keep[k]], want[k][keep[k]], norm[k][keep[k]], t, k)
        else:
            compare(v, want[k], norm[k], t, k)
    return Yt, dXt, dW, db


PATTERNS = [(1, 0), (2, 0), (2, 1), (3, 2), (5, 1), (16, 9), (40, 39)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_tiny_all_pattern_pairs(dtype):
    X, W, b, dY = make_inputs(dtype, 5, 13, 11, seed=1805)
    for i, (pin, pout) in enumerate(itertools.product(PATTERNS, repeat=2)):
        for act in ("none", "relu"):
            run_layer(dtype, X, W, b, dY, pin, pout, act, 1.0 / 0.7, api.ARD_DROPPED_ZERO, lists=i % 2 == 0)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(200, 300, 260), (130, 1000, 70), (64, 96, 520), (8, 4104, 36), (1, 130, 70)])
def test_multi_tile_ragged(dtype, shape):
    B, K, N = shape
    X, W, b, dY = make_inputs(dtype, B, K, N, seed=sum(shape))
    for i, (pin, pout, act) in enumerate([((3, 1), (2, 0), "relu"), ((1, 0), (5, 4), "none"),
                                          ((4, 2), (1, 0), "relu"), ((7, 0), (3, 1), "none")]):
        run_layer(dtype, X, W, b, dY, pin, pout, act, 1.25, api.ARD_DROPPED_ZERO,
                  use_null_plans=False, lists=i % 2 == 1)


@pytest.mark.parametrize("B", [16, 20, 32])
def test_small_batch_tall_layer_fp32(B):
    """At most 32 batch columns and 161 row tiles of 128 rows: the fp32
    forward runs on 128 x 32 tiles (ragged rows and columns)."""
    K, N = 264, 128 * 160 + 37
    X, W, b, dY = make_inputs("f32", B, K, N, seed=B)
    for pin, act in (((1, 0), "relu"), ((2, 1), "none")):
        run_layer("f32", X, W, b, dY, pin, (1, 0), act, 1.25, api.ARD_DROPPED_ZERO, use_null_plans=False)


def random_cases(dtype, n, seed):
    """n seeded layer shapes and patterns spread over the planner's choices:
    batch from 1 to 600, sides from 1 to 3000 (the long contractions take a
    k split), periods 1 to 16 with any offset, both activations and modes."""
    rng = np.random.default_rng(seed)
    cases = []
    for _ in range(n):
        B = int(rng.choice([1, 16, 64, 96, 128, 200, 256, 512, 600]))
        K = int(rng.integers(1, 3001))
        N = int(rng.integers(1, 3001))
        pin = (1, 0) if rng.random() < 0.3 else (lambda q: (q, int(rng.integers(0, q))))(int(rng.integers(2, 17)))
        pout = (1, 0) if rng.random() < 0.3 else (lambda q: (q, int(rng.integers(0, q))))(int(rng.integers(2, 17)))
        act = "relu" if rng.random() < 0.5 else "none"
        dropped = api.ARD_DROPPED_SKIP if rng.random() < 0.5 else api.ARD_DROPPED_ZERO
        cases.append((B, K, N, pin, pout, act, dropped))
    return cases


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_random_shapes_and_patterns(dtype):
    """Every product of 12 random layers (see random_cases) against the oracle,
    with the sentinel checks of SKIP mode; the case is printed before it runs."""
    for i, (B, K, N, pin, pout, act, dropped) in enumerate(random_cases(dtype, 12, 8939 + (dtype == "bf16"))):
        print(f"case {i}: {dtype} B={B} K={K} N={N} pin={pin} pout={pout} act={act} dropped={dropped}", flush=True)
        X, W, b, dY = make_inputs(dtype, B, K, N, seed=1805 + i)
        sentinel = -3.25 if dropped == api.ARD_DROPPED_SKIP else None
        run_layer(dtype, X, W, b, dY, pin, pout, act, 1.0 / 0.7, dropped, use_null_plans=i % 3 != 0,
                  sentinel=sentinel, lists=i % 2 == 0)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape,pin", [((64, 96, 520), (3, 1)), ((200, 1000, 260), (2, 0)), ((128, 2048, 1024), (7, 4)),
                                       ((8, 130, 70), (1, 0)), ((256, 600, 2048), (16, 15))])
def test_input_major_weights(dtype, shape, pin):
    """A last layer (every output kept) with W stored input-major, W^T[K][N]:
    fwd, bwd_data, bwd_weight (dW^T), the one-call backward and the momentum
    update against the oracle on W, in both dropped modes; dropped input rows
    of dW^T keep a sentinel in SKIP mode and are 0 in ZERO mode."""
    B, K, N = shape
    X, W, b, dY = make_inputs(dtype, B, K, N, seed=sum(shape) + pin[0])
    m_in = opat.row_mask(K, *pin)
    m_out = np.ones(N)
    in_plan = row_plan(K, *pin, with_list=False) if pin != (1, 0) else None
    Y64 = ofc.fc_forward(f64(X), f64(W), f64(b), m_in, m_out, 1.25, "relu")
    Ys = synth.to_storage(torch.from_numpy(Y64).float(), dtype)
    dX64, dW64, db64 = ofc.fc_backward(f64(X), f64(W), f64(Ys), f64(dY), m_in, m_out, 1.25, "relu")
    Xa, Wa = np.abs(f64(X) * m_in[None, :]), np.abs(f64(W))
    G = ofc.fc_output_grad(f64(Ys), f64(dY), m_out, 1.25, "relu")
    t = tol(dtype)
    Xt, WTd, dYt, Yst = to_dev(X.T), to_dev(W.T.contiguous()), to_dev(dY.T), to_dev(Ys.T)
    sdt = synth.storage_dtype(dtype)
    for dropped, fill in ((api.ARD_DROPPED_SKIP, -3.25), (api.ARD_DROPPED_ZERO, 0.0)):
        desc = api.fc_desc(ard_dtype(dtype), B, K, N, in_plan, None, 1.25, api.ARD_ACT_RELU, dropped,
                           api.ARD_WEIGHTS_INPUT_MAJOR)
        ws = workspace(api.ard_fc_workspace_bytes(desc))
        Yt = torch.full((N, B), 9.0, dtype=sdt, device=device())
        dXt = torch.full((K, B), fill, dtype=sdt, device=device())
        dWT = torch.full((K, N), fill, dtype=torch.float32, device=device())
        db = torch.full((N,), fill, dtype=torch.float32, device=device())
        api.ard_fc_fwd(desc, Xt, WTd, to_dev(b), Yt, ws)
        api.ard_fc_bwd_data(desc, dYt, Yst, WTd, dXt, ws)
        api.ard_fc_bwd_weight(desc, Xt, dYt, Yst, dWT, db, ws)
        dXt2, dWT2, db2 = (torch.full_like(x, fill) for x in (dXt, dWT, db))
        api.ard_fc_bwd(desc, Xt, dYt, Yst, WTd, dXt2, dWT2, db2, ws)
        torch.cuda.synchronize()
        assert torch.equal(dXt2, dXt) and torch.equal(dWT2, dWT) and torch.equal(db2, db)
        compare(f64(Yt).T, Y64, 1.25 * (Xa @ Wa.T + np.abs(f64(b))[None, :]), t, "Y")
        keep = m_in > 0
        got_dX, got_dW = f64(dXt).T, f64(dWT).T
        compare(got_dX[:, keep], dX64[:, keep], 1.25 * (np.abs(G) @ Wa)[:, keep], t, "dX")
        compare(got_dW[:, keep], dW64[:, keep], 1.25 * (np.abs(G).T @ Xa)[:, keep], t, "dW")
        compare(f64(db), db64, 1.25 * np.abs(G).sum(0), t, "db")
        assert (got_dX[:, ~keep] == fill).all() and (got_dW[:, ~keep] == fill).all(), "dropped inputs"
        if dropped == api.ARD_DROPPED_SKIP:
            # the momentum update on the kept input rows of W^T (all outputs)
            V = torch.full((K, N), 0.5, device=device())
            Vb = torch.full((N,), 0.25, device=device())
            bias = to_dev(b)
            W0, V0, bias0, Vb0 = WTd.clone(), V.clone(), bias.clone(), Vb.clone()
            api.ard_fc_sgd_momentum(desc, WTd, V, dWT, bias, Vb, db, 0.01, 0.9)
            torch.cuda.synchronize()
            Wn, Vn, bn, Vbn = ofc.sgd_momentum(f64(W0).T, f64(V0).T, f64(dWT).T, m_out, m_in, 0.01, 0.9,
                                               f64(bias0), f64(Vb0), f64(db))
            kw = np.outer(m_out, m_in) > 0
            compare(f64(V).T[kw], Vn[kw], (0.9 * np.abs(f64(V0).T) + np.abs(f64(dWT).T) + 1.0)[kw], F32_TOL_UPD,
                    "V")
            compare(f64(WTd).T[kw], Wn[kw], (np.abs(Wn) + 0.01 * np.abs(Vn) + 1e-3)[kw], t, "W")
            compare(f64(Vb), Vbn, 0.9 * np.abs(f64(Vb0)) + np.abs(f64(db)) + 1.0, F32_TOL_UPD, "Vb")
            compare(f64(bias), bn, np.abs(bn) + 0.01 * np.abs(Vbn) + 1e-3, F32_TOL_UPD, "b")
            assert np.array_equal(f64(WTd).T[~kw], f64(W0).T[~kw]) and np.array_equal(f64(V).T[~kw], f64(V0).T[~kw])
            WTd.copy_(W0)
    # an output pattern cannot be read from input-major rows; no compact copy exists
    bad = api.fc_desc(ard_dtype(dtype), B, K, N, in_plan, row_plan(N, 2, 1, with_list=False), 1.0,
                      api.ARD_ACT_NONE, api.ARD_DROPPED_SKIP, api.ARD_WEIGHTS_INPUT_MAJOR)
    with pytest.raises(RuntimeError, match="UNSUPPORTED|every output"):
        api.ard_fc_fwd(bad, Xt, WTd, None, torch.empty((N, B), dtype=sdt, device=device()),
                       workspace(1 << 20))
    good = api.fc_desc(ard_dtype(dtype), B, K, N, in_plan, None, 1.0, api.ARD_ACT_NONE, api.ARD_DROPPED_SKIP,
                       api.ARD_WEIGHTS_INPUT_MAJOR)
    with pytest.raises(RuntimeError, match="compact"):
        api.ard_fc_compact_weights(good, WTd, torch.empty(K * N, dtype=sdt, device=device()))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_skip_mode_leaves_dropped_entries_untouched(dtype):
    X, W, b, dY = make_inputs(dtype, 96, 160, 144, seed=7)
    run_layer(dtype, X, W, b, dY, (3, 0), (2, 1), "relu", 2.0, api.ARD_DROPPED_SKIP, sentinel=-7.5)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_dropped_data_never_enter_the_arithmetic(dtype):
    X, W, b, dY = make_inputs(dtype, 80, 192, 176, seed=11)
    run_layer(dtype, X, W, b, dY, (4, 3), (3, 1), "relu", 1.0, api.ARD_DROPPED_ZERO, poison=True)
    run_layer(dtype, X, W, b, dY, (2, 0), (5, 2), "none", 1.0, api.ARD_DROPPED_SKIP, poison=True,
              sentinel=3.0)


def test_single_fc_layer_fp32_full_config():
    """Single FC layer fp32: X[64x784] ~ N(0,1), W (512 outputs x 784) ~ N(0, 0.05^2),
    row dropout of the 512 outputs with period 2 and a seeded offset, dY ~ N(0,1)."""
    X, W, _, dY = make_inputs("f32", 64, 784, 512, seed=1805, w_std=0.05, bias=False)
    K2 = np.zeros(16)
    K2[1] = 1.0
    per, off = oprng.sample_row_pattern(K2, 8939, 0, 0)
    assert per == 2
    run_layer("f32", X, W, None, dY, (1, 0), (per, off), "none", 1.0, api.ARD_DROPPED_ZERO)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_bitwise_deterministic(dtype):
    X, W, b, dY = make_inputs(dtype, 256, 384, 320, seed=3)
    r1 = run_layer(dtype, X, W, b, dY, (3, 2), (2, 0), "relu", 1.0, api.ARD_DROPPED_ZERO)
    r2 = run_layer(dtype, X, W, b, dY, (3, 2), (2, 0), "relu", 1.0, api.ARD_DROPPED_ZERO)
    for a, c in zip(r1, r2):
        assert torch.equal(a, c)


def test_invalid_arguments_are_rejected_before_launch():
    d = device()
    X = torch.zeros(16, 8, device=d)
    W = torch.zeros(8, 16, device=d)
    Y = torch.zeros(8, 8, device=d)
    plan_bad = row_plan(10, 2, 1)  # covers 10 neurons, the layer has 8 outputs
    for desc in (api.fc_desc(api.ARD_F32, 0, 16, 8), api.fc_desc(7, 8, 16, 8),
                 api.fc_desc(api.ARD_F32, 8, 16, 8, out_plan=plan_bad),
                 api.fc_desc(api.ARD_F32, 8, 16, 8, act=5),
                 api.fc_desc(api.ARD_F32, 8, 16, 8, scale=float("inf"))):
        with pytest.raises(api.ArdError):
            api.ard_fc_fwd(desc, X, W, None, Y)
    good = api.fc_desc(api.ARD_F32, 8, 16, 8)
    with pytest.raises(api.ArdError):
        api.ard_fc_fwd(good, None, W, None, Y)
    # a layer whose small output grid splits the contraction needs its workspace
    big_k = api.fc_desc(api.ARD_F32, 8, 4096, 8)
    assert api.ard_fc_workspace_bytes(big_k) > 0
    Xk, Wk = torch.zeros(4096, 8, device=d), torch.zeros(8, 4096, device=d)
    with pytest.raises(api.ArdError) as e:
        api.ard_fc_fwd(big_k, Xk, Wk, None, Y)
    assert e.value.status == 5
    with pytest.raises(api.ArdError):
        api.ard_fc_fwd(api.fc_desc(api.ARD_F32, 8, 16, 8, weight_layout=7), X, W, None, Y)
    with pytest.raises(api.ArdError):
        api.ard_fc_fwd(good, X[:, 1:].contiguous().view(-1)[1:], W, None, Y)  # misaligned
    relu = api.fc_desc(api.ARD_F32, 8, 16, 8, act=api.ARD_ACT_RELU)
    with pytest.raises(api.ArdError):  # misaligned input gate
        api.ard_fc_bwd_data(relu, Y, None, W, X, Xgate=X.view(-1)[1:])


@pytest.mark.parametrize("shape,pin,pout", [
    ((256, 1000, 520), (3, 1), (2, 0)),     # gathers both sides, K tail, ragged tiles
    ((512, 2048, 1536), (1, 0), (5, 4)),    # one-sided, several 256-wide tiles
    ((128, 4096, 64), (2, 1), (1, 0)),      # tiny output grid: split contraction
    ((1024, 512, 640), (7, 3), (3, 2)),     # batch-heavy
])
def test_bf16_large_tiles(shape, pin, pout):
    B, K, N = shape
    X, W, b, dY = make_inputs("bf16", B, K, N, seed=B + K)
    run_layer("bf16", X, W, b, dY, pin, pout, "relu", 1.0, api.ARD_DROPPED_SKIP, use_null_plans=False,
              sentinel=-3.0)
    run_layer("bf16", X, W, b, dY, pin, pout, "none", 2.0, api.ARD_DROPPED_ZERO)


@pytest.mark.parametrize("dtype,B,K,N,pout", [
    ("f32", 128, 1024, 1024, (1, 0)),   # 64x64 tiles: one wave per output block, no k split
    ("f32", 96, 2048, 2048, (3, 1)),    # 128x128 tiles
    ("f32", 256, 300, 260, (2, 1)),     # 32x32 tiles, k split over 8 waves, ragged rows
    ("f32", 8192, 64, 72, (1, 0)),      # contraction split over workgroups: separate bias kernel
    ("bf16", 256, 1024, 2048, (5, 4)),  # large bf16 tiles
    ("bf16", 128, 96, 100, (1, 0)),     # bf16 32x32 tiles, k split over 4 waves
    ("bf16", 4096, 64, 64, (2, 0)),     # bf16 split contraction
])
def test_bias_gradient_with_the_weight_gradient(dtype, B, K, N, pout):
    """dbias of an ungated layer comes from the row sums of the weight-gradient
    product's first operand on every tile configuration without a k split,
    and from its own kernel otherwise; both against the oracle."""
    X, W, b, dY = make_inputs(dtype, B, K, N, seed=B + N)
    run_layer(dtype, X, W, b, dY, (1, 0), pout, "none", 1.5, api.ARD_DROPPED_ZERO, use_null_plans=False)
    run_layer(dtype, X, W, b, dY, (1, 0), pout, "none", 1.0, api.ARD_DROPPED_SKIP, use_null_plans=False,
              sentinel=-2.0)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_pregated_gradient_and_input_gate(dtype):
    """Yt = NULL takes dYt as already gated; Xgate gates dXt with [Xgate > 0]."""
    B, K, N = 128, 264, 192
    X, W, b, dY = make_inputs(dtype, B, K, N, seed=99)
    Xr = synth.to_storage(torch.relu(X.float()), dtype)           # a ReLU output as this layer's input
    m_in, m_out = opat.row_mask(K, 3, 1), opat.row_mask(N, 2, 0)
    Y64 = ofc.fc_forward(f64(Xr), f64(W), f64(b), m_in, m_out, 1.0, "relu")
    Ys = synth.to_storage(torch.from_numpy(Y64).float(), dtype)
    G = synth.to_storage(torch.from_numpy(ofc.fc_output_grad(f64(Ys), f64(dY), m_out, 1.0, "relu")).float(),
                         dtype)  # exact: dY times a 0/1 gate
    dX64, dW64, db64 = ofc.fc_backward(f64(Xr), f64(W), f64(Ys), f64(dY), m_in, m_out, 1.0, "relu")
    in_plan, out_plan = row_plan(K, 3, 1), row_plan(N, 2, 0)
    desc = api.fc_desc(ard_dtype(dtype), B, K, N, in_plan, out_plan, 1.0, api.ARD_ACT_RELU, api.ARD_DROPPED_ZERO)
    ws = workspace(api.ard_fc_workspace_bytes(desc))
    Xt, Wd, Gt, Xrt = to_dev(X.T), to_dev(W), to_dev(G.T), to_dev(Xr.T)
    sdt = synth.storage_dtype(dtype)
    dXt = torch.empty(K, B, dtype=sdt, device=device())
    dW = torch.empty(N, K, device=device())
    db = torch.empty(N, device=device())
    api.ard_fc_bwd_data(desc, Gt, None, Wd, dXt, ws, Xgate=Xrt)
    api.ard_fc_bwd_weight(desc, Xrt, Gt, None, dW, db, ws)
    torch.cuda.synchronize()
    Ga = np.abs(f64(G))
    ndX = (Ga @ np.abs(f64(W))) * m_in[None, :]
    want_dX = dX64 * (f64(Xr) > 0)
    compare(f64(dXt).T, want_dX, ndX * (f64(Xr) > 0), tol(dtype), "dX gated")
    compare(f64(dW), dW64, (Ga.T @ np.abs(f64(Xr))) * np.outer(m_out, m_in), tol(dtype), "dW")
    compare(f64(db), db64, Ga.sum(0), tol(dtype), "db")


@pytest.mark.parametrize("dtype,B,K,N,pats", [
    ("bf16", 2048, 8192, 8192, ((3, 2), (2, 1))),
    # dense, 256 x 256 output tiles in all three passes, a partial last K slab
    # (8152 = 254 * 32 + 24) and a ragged last tile row
    ("bf16", 2048, 8152, 8192, ((1, 0), (1, 0))),
    # fp32 128 x 128 tiles (fwd, bwd_weight) with a partial last K slab
    ("f32", 1024, 2040, 4096, ((1, 0), (1, 0))),
    ("f32", 1024, 2040, 4096, ((2, 1), (3, 0))),
    # bf16 tile configurations and split-K paths the planner takes for these
    # shapes: 128x128 tiles split 4 (fwd), 128x256 tiles split 16 (bwd_data)
    ("bf16", 256, 1024, 2048, ((3, 0), (1, 0))),
    # 256x256 tiles split 4 (fwd, bwd_data)
    ("bf16", 512, 8192, 8192, ((1, 0), (1, 0))),
    # 256x128 tiles split 4 (bwd_weight)
    ("bf16", 2048, 1024, 4096, ((3, 0), (1, 0))),
    # 32x32 tiles split 4 (bwd_data)
    ("bf16", 256, 1024, 2048, ((4, 1), (1, 0))),
    # fp32 32x32 tiles (8 waves) and the fp32 split-K path of a long contraction (fwd)
    ("f32", 128, 16384, 256, ((1, 0), (1, 0))),
], ids=["bf16-patterned", "bf16-dense-ragged", "f32-dense-ragged", "f32-patterned", "bf16-t128-split",
        "bf16-t256-split", "bf16-t256x128-split", "bf16-t32-split", "f32-t32-split"])
def test_wide_layer_full_size_sampled(dtype, B, K, N, pats):
    """One hidden layer of the wide MLP in the launch configuration of the
    benchmark (compact weights, SKIP, workspace), against the oracle on sampled
    rows and columns. The oracle's forward output, rounded to the storage type,
    is the ReLU gate of both backward implementations."""
    g = synth.generator(1805 + 4)
    X = synth.to_storage(torch.relu(synth.normal(g, (B, K))), dtype)
    W = synth.to_storage(synth.he(g, N, K), dtype)
    dY = synth.to_storage(synth.normal(g, (B, N)), dtype)
    (pi, oi), (po, oo) = pats
    m_in, m_out = opat.row_mask(K, pi, oi), opat.row_mask(N, po, oo)
    Xf, Wf, dYf = f64(X), f64(W), f64(dY)
    Y64 = ofc.fc_forward(Xf, Wf, None, m_in, m_out, 1.0, "relu")
    Ys = synth.to_storage(torch.from_numpy(Y64).float(), dtype)
    in_plan, out_plan = row_plan(K, pi, oi), row_plan(N, po, oo)
    desc = api.fc_desc(ard_dtype(dtype), B, K, N, in_plan, out_plan, 1.0, api.ARD_ACT_RELU, api.ARD_DROPPED_SKIP,
                       api.ARD_WEIGHTS_COMPACT)
    Xt, Wd, dYt, Yst = to_dev(X.T), to_dev(W), to_dev(dY.T), to_dev(Ys.T)
    sdt = synth.storage_dtype(dtype)
    Wc = torch.empty(api.ard_fc_compact_bytes(desc) // Wd.element_size(), dtype=sdt, device=device())
    api.ard_fc_compact_weights(desc, Wd, Wc)
    ws = workspace(api.ard_fc_workspace_bytes(desc))
    Yt = torch.zeros(N, B, dtype=sdt, device=device())
    dXt = torch.zeros(K, B, dtype=sdt, device=device())
    dW = torch.zeros(N, K, device=device())
    api.ard_fc_fwd(desc, Xt, Wc, None, Yt, ws)
    api.ard_fc_bwd_data(desc, dYt, Yst, Wc, dXt, ws)
    api.ard_fc_bwd_weight(desc, Xt, dYt, Yst, dW, None, ws)
    torch.cuda.synchronize()
    rng = np.random.default_rng(1)
    Sin, Sout = np.array(opat.row_kept_list(K, pi, oi)), np.array(opat.row_kept_list(N, po, oo))
    rows = np.sort(rng.choice(Sout, 40, replace=False))
    cols = np.sort(rng.choice(Sin, 40, replace=False))
    Xm = Xf * m_in[None, :]
    compare(f64(Yt)[rows].T, Y64[:, rows], np.abs(Xm) @ np.abs(Wf[rows]).T, tol(dtype), "Y rows")
    G = ofc.fc_output_grad(f64(Ys), dYf, m_out, 1.0, "relu")        # [B][N]
    Wk = Wf[:, cols] * m_out[:, None]
    compare(f64(dXt)[cols].T, G @ Wk, np.abs(G) @ np.abs(Wk), tol(dtype), "dX cols")
    compare(f64(dW)[np.ix_(rows, cols)], G[:, rows].T @ Xf[:, cols],
            np.abs(G[:, rows]).T @ np.abs(Xf[:, cols]), tol(dtype), "dW")
    # every output tile: Y in full (normwise), dX and dW through random projections
    Yg = f64(Yt)
    err = np.abs(Yg[Sout] - Y64.T[Sout]).max() / np.abs(Y64).max()
    assert err <= tol(dtype), f"Y normwise error {err:.3e}"
    v, u = rng.standard_normal(B), rng.standard_normal(K)
    Wm = Wf * m_out[:, None]
    compare(f64(dXt)[Sin] @ v, (Wm[:, Sin].T @ (G.T @ v)), np.abs(Wm[:, Sin]).T @ (np.abs(G).T @ np.abs(v)),
            tol(dtype), "dX projection")
    dWg = f64(dW)
    compare(dWg[np.ix_(Sout, Sin)] @ u[Sin], G[:, Sout].T @ (Xf[:, Sin] @ u[Sin]),
            np.abs(G[:, Sout]).T @ (np.abs(Xf[:, Sin]) @ np.abs(u[Sin])), tol(dtype), "dW projection")
    dropped_rows = np.setdiff1d(np.arange(N), Sout)[:64]
    assert not Yg[dropped_rows].any() and not dWg[dropped_rows].any()


@pytest.mark.parametrize("B,K,N,pin,pout", [
    (128, 784, 2048, (2, 1), (2, 0)),     # 32x32 tiles (fwd and bwd_data), K tail
    (512, 1000, 2600, (3, 1), (2, 1)),    # 64x64 tiles (fwd), ragged
    (1024, 5120, 2600, (2, 1), (2, 0)),   # 64x64 (fwd) and 128x128 tiles (bwd_data)
    (1024, 1536, 5200, (5, 3), (2, 1)),   # 128x128 tiles (fwd)
], ids=["t32", "t64", "t128-bwd", "t128-fwd"])
def test_fp32_full_weights_with_input_gather(B, K, N, pin, pout):
    """fp32 layers given the full W with a gathered input side (the compact
    copy built in the workspace): fwd and the pre-gated bwd_data with an input
    gate on every fp32 tile configuration, against the oracle on sampled
    neurons over the whole batch and on sampled batch entries over every
    output tile. Dropped input columns of W hold NaN and are never read."""
    g = synth.generator(K + N)
    X = torch.relu(synth.normal(g, (B, K)))
    W = synth.normal(g, (N, K), 0.05)
    b = synth.normal(g, (N,), 0.1)
    dY = synth.normal(g, (B, N))
    (pi, oi), (po, oo) = pin, pout
    m_in, m_out = opat.row_mask(K, pi, oi), opat.row_mask(N, po, oo)
    in_plan, out_plan = row_plan(K, pi, oi), row_plan(N, po, oo)
    args = (api.ARD_F32, B, K, N, in_plan, out_plan, 1.0, api.ARD_ACT_RELU, api.ARD_DROPPED_ZERO)
    desc = api.fc_desc(*args)
    ws = workspace(api.ard_fc_workspace_bytes(desc))
    Xt, Wd, dYt, bd = to_dev(X.T), to_dev(W), to_dev(dY.T), to_dev(b)
    Wd[:, torch.from_numpy(m_in == 0).to(device())] = float("nan")  # dropped columns are never read
    Yt = torch.full((N, B), 5.0, device=device())
    dXt = torch.full((K, B), 5.0, device=device())
    api.ard_fc_fwd(desc, Xt, Wd, bd, Yt, ws)
    api.ard_fc_bwd_data(desc, dYt, None, Wd, dXt, ws, Xgate=Xt)
    torch.cuda.synchronize()
    Xf, Wf, bf, dYf = f64(X), f64(W), f64(b), f64(dY)
    Sin, Sout = np.array(opat.row_kept_list(K, pi, oi)), np.array(opat.row_kept_list(N, po, oo))
    rng = np.random.default_rng(5)
    rows = np.sort(rng.choice(Sout, min(48, len(Sout)), replace=False))
    cols = np.sort(rng.choice(Sin, min(48, len(Sin)), replace=False))
    bs = np.sort(rng.choice(B, 16, replace=False))
    Yg, dXg = f64(Yt).T, f64(dXt).T
    Xa, Wa = np.abs(Xf * m_in[None, :]), np.abs(Wf)

    def dx_oracle(xs, ws_cols, dys, mi):
        # the oracle's bwd_data of the pre-gated gradient, then the ReLU gate of the layer below
        dX = ofc.fc_backward(xs, ws_cols, None, dys, mi, m_out, 1.0, "none")[0]
        return ofc.fc_output_grad(xs, dX, np.ones(dX.shape[1]), 1.0, "relu")

    # sampled neurons over the whole batch
    compare(Yg[:, rows], ofc.fc_forward(Xf, Wf[rows], bf[rows], m_in, m_out[rows], 1.0, "relu"),
            Xa @ Wa[rows].T + np.abs(bf[rows])[None, :], tol("f32"), "Y rows")
    Wo = Wa * m_out[:, None]
    compare(dXg[:, cols], dx_oracle(Xf[:, cols], Wf[:, cols], dYf, m_in[cols]),
            np.abs(dYf) @ Wo[:, cols], tol("f32"), "dX cols")
    # sampled batch entries over every output tile
    keep_out, keep_in = m_out > 0, m_in > 0
    compare(Yg[bs][:, keep_out], ofc.fc_forward(Xf[bs], Wf, bf, m_in, m_out, 1.0, "relu")[:, keep_out],
            (Xa[bs] @ Wa.T + np.abs(bf)[None, :])[:, keep_out], tol("f32"), "Y batch rows")
    compare(dXg[bs][:, keep_in], dx_oracle(Xf[bs], Wf, dYf[bs], m_in)[:, keep_in],
            (np.abs(dYf[bs]) @ Wo)[:, keep_in], tol("f32"), "dX batch rows")
    Yg, dXg = Yg.T, dXg.T
    assert not Yg[np.setdiff1d(np.arange(N), Sout)].any() and not dXg[np.setdiff1d(np.arange(K), Sin)].any()



@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_compact_weights_batch(dtype):
    """One launch for several layers' compact weights: each equals the gather
    W[S_out][S_in] (padding columns 0), bitwise the single-layer call."""
    d = device()
    sdt = synth.storage_dtype(dtype)
    layers = [(130, 70, (3, 1), (2, 0)), (10, 2048, (5, 4), (1, 0)), (4104, 36, (1, 0), (7, 3))]
    descs, Ws, Wcs, singles = [], [], [], []
    for i, (K, N, pin, pout) in enumerate(layers):
        g = synth.generator(40 + i)
        W = synth.to_storage(synth.normal(g, (N, K)), dtype)
        desc = api.fc_desc(ard_dtype(dtype), 8, K, N, row_plan(K, *pin, with_list=False),
                           row_plan(N, *pout, with_list=False), 1.0, api.ARD_ACT_NONE, api.ARD_DROPPED_SKIP,
                           api.ARD_WEIGHTS_COMPACT)
        n = max(api.ard_fc_compact_bytes(desc) // (2 if dtype == "bf16" else 4), 1)
        Wc = torch.full((n,), 5.0, dtype=sdt, device=d)
        one = torch.full((n,), 5.0, dtype=sdt, device=d)
        api.ard_fc_compact_weights(desc, to_dev(W), one)
        descs.append(desc)
        Ws.append(to_dev(W))
        Wcs.append(Wc)
        singles.append((one, W, K, N, pin, pout, api.ard_fc_compact_ld(desc)))
    batch = api.CompactBatch(descs, Ws, Wcs)
    api.ard_fc_compact_weights_batch(batch)
    torch.cuda.synchronize()
    for Wc, (one, W, K, N, pin, pout, ldc) in zip(Wcs, singles):
        assert torch.equal(Wc, one)
        Sin, Sout = opat.row_kept_list(K, *pin), opat.row_kept_list(N, *pout)
        got = f64(Wc[:len(Sout) * ldc].view(len(Sout), ldc))
        assert np.array_equal(got[:, :len(Sin)], f64(W)[np.ix_(Sout, Sin)])
        assert not got[:, len(Sin):].any()
    with pytest.raises(api.ArdError):
        api.ard_fc_compact_weights_batch(api.CompactBatch(descs * 2, Ws * 2, Wcs * 2))  # 6 > 4 layers
    other = api.fc_desc(api.ARD_BF16 if dtype == "f32" else api.ARD_F32, 8, 130, 70)
    with pytest.raises(api.ArdError):
        api.ard_fc_compact_weights_batch(api.CompactBatch([descs[0], other], Ws[:2], Wcs[:2]))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("pin,pout", [((1, 0), (1, 0)), ((3, 1), (2, 0)), ((5, 4), (1, 0))])
def test_sgd_momentum_against_oracle(dtype, pin, pout):
    """Two momentum-SGD steps restricted to the kept weights: kept entries
    match the oracle, dropped weights, momentum and bias entries are untouched
    bit for bit."""
    d = device()
    N, K, lr, mu = 130, 260, 0.01, 0.9
    g = synth.generator(77)
    W = synth.to_storage(synth.normal(g, (N, K)), dtype)
    V, b, Vb = synth.normal(g, (N, K), 0.1), synth.normal(g, (N,)), synth.normal(g, (N,), 0.1)
    desc = api.fc_desc(ard_dtype(dtype), 8, K, N, row_plan(K, *pin, with_list=False),
                       row_plan(N, *pout, with_list=False), 1.0, api.ARD_ACT_NONE, api.ARD_DROPPED_SKIP)
    Wd, Vd, bd, Vbd = to_dev(W), to_dev(V), to_dev(b), to_dev(Vb)
    m_out, m_in = opat.row_mask(N, *pout), opat.row_mask(K, *pin)
    Wo, Vo, bo, Vbo = f64(W), f64(V), f64(b), f64(Vb)
    for step in range(2):
        dW, db = synth.normal(g, (N, K)), synth.normal(g, (N,))
        api.ard_fc_sgd_momentum(desc, Wd, Vd, to_dev(dW), bd, Vbd, to_dev(db), lr, mu)
        torch.cuda.synchronize()
        # from the second step on the oracle continues from the stored weights
        # (bf16 rounds them each step)
        Wo, Vo, bo, Vbo = ofc.sgd_momentum(Wo, Vo, f64(dW), m_out, m_in, lr, mu, bo, Vbo, f64(db))
        keep = np.outer(m_out, m_in) > 0
        compare(f64(Vd)[keep], Vo[keep], (mu * np.abs(Vo) + np.abs(f64(dW)) + 1.0)[keep], F32_TOL_UPD, "V")
        compare(f64(Wd)[keep], Wo[keep], (np.abs(Wo) + lr * np.abs(Vo) + 1e-3)[keep], tol(dtype), "W")
        compare(f64(bd), bo, np.abs(bo) + lr * np.abs(Vbo) + 1e-3, F32_TOL_UPD, "b")
        assert np.array_equal(f64(Wd)[~keep], f64(W)[~keep]) and np.array_equal(f64(Vd)[~keep], f64(V)[~keep])
        assert np.array_equal(f64(bd)[m_out == 0], f64(b)[m_out == 0])
        Wo = np.where(keep, f64(Wd), Wo)
    with pytest.raises(api.ArdError):
        api.ard_fc_sgd_momentum(desc, Wd, Vd, to_dev(dW), bd, None, to_dev(db), lr, mu)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("pin,pout", [((1, 0), (1, 0)), ((3, 1), (2, 0)), ((5, 4), (1, 0)), ((2, 0), (7, 6))])
def test_sgd_momentum_compact_gradient(dtype, pin, pout):
    """The update fed the compact gradient dWc[kept_out][ldc] (layout
    ARD_WEIGHTS_COMPACT_GRAD) equals, bit for bit, the update fed the same
    values in the full layout."""
    d = device()
    N, K, lr, mu = 130, 260, 0.01, 0.9
    g = synth.generator(78)
    W = synth.to_storage(synth.normal(g, (N, K)), dtype)
    V, b, Vb = synth.normal(g, (N, K), 0.1), synth.normal(g, (N,)), synth.normal(g, (N,), 0.1)
    dW, db = synth.normal(g, (N, K)), synth.normal(g, (N,))
    args = (ard_dtype(dtype), 8, K, N, row_plan(K, *pin, with_list=False), row_plan(N, *pout, with_list=False), 1.0,
            api.ARD_ACT_NONE, api.ARD_DROPPED_SKIP)
    full, comp = api.fc_desc(*args), api.fc_desc(*args, api.ARD_WEIGHTS_COMPACT_GRAD)
    Sin, Sout = opat.row_kept_list(K, *pin), opat.row_kept_list(N, *pout)
    ldc = api.ard_fc_compact_ld(comp)
    dWc = torch.full((len(Sout), ldc), float("nan"))
    dWc[:, :len(Sin)] = dW[Sout][:, Sin]
    outs = []
    for desc, grad in ((full, dW), (comp, dWc)):
        Wd, Vd, bd, Vbd = to_dev(W), to_dev(V), to_dev(b), to_dev(Vb)
        api.ard_fc_sgd_momentum(desc, Wd, Vd, to_dev(grad), bd, Vbd, to_dev(db), lr, mu)
        outs.append((Wd, Vd, bd, Vbd))
    torch.cuda.synchronize()
    for a, c in zip(*outs):
        assert torch.equal(a, c)
