"""Host side of the C ABI (no GPU needed): exported symbols, the sampler and
bitmaps bit-exact against the oracle, the Alg. 1 search against the oracle's
closed-form minimiser, and argument validation."""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import patterns as opat
from oracle import prng as oprng
from oracle import search as osearch
from paper_1805_08939_amd import _ffi, api

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "ard.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"\b(ard_[a-z0-9_]+)\s*\(", text)
    return sorted(set(names))


def test_library_exports_every_declared_function():
    L = ctypes.CDLL(_ffi.LIB_PATH)
    names = declared_functions()
    assert len(names) >= 20
    for name in names:
        assert hasattr(L, name), name
    assert set(names) == set(_ffi.SIGNATURES), "binding and header disagree"


def test_version_and_status_strings():
    assert api.ard_version() == 3
    assert api.ard_status_string(0) == "ARD_OK"
    assert api.ard_status_string(4) == "ARD_ERR_NOT_CONVERGED"


def _k_cases():
    cases = [osearch.closed_form(p, 16) for p in (0.3, 0.5, 0.7)]
    cases.append(osearch.distribution_for_rate(0.0, 16))
    e = np.zeros(9)
    e[6] = 1.0
    cases.append(e)
    # entries that leave the running sum below 1: exercises the fallback
    cases.append(np.array([0.2, 0.0, 0.3, 0.4999999999, 0.0]))
    cases.append(np.array([1e-300, 0.5, 1e-17, 0.5 - 1e-16]))
    cases.append(osearch.closed_form(0.6, 64))
    return cases


@pytest.mark.parametrize("case", range(8))
def test_sampler_bit_exact_against_oracle(case):
    K = _k_cases()[case]
    rng = np.random.default_rng(case)
    n = 15_000
    seeds = rng.integers(0, 2**63, size=n, dtype=np.uint64)
    streams = rng.integers(0, 2**24, size=n)
    iters = rng.integers(0, 2**40, size=n)
    for s, st, it in zip(seeds.tolist(), streams.tolist(), iters.tolist()):
        assert api.ard_sample_row_pattern(K, s, st, it) == oprng.sample_row_pattern(K, s, st, it)
    for it in range(2000):  # consecutive iterations of one layer stream
        assert api.ard_sample_row_pattern(K, 8939, 1, it) == oprng.sample_row_pattern(K, 8939, 1, it)


def test_bitmaps_bit_exact_against_oracle():
    for tn, tk in [(1, 1), (3, 5), (64, 64), (7, 33)]:
        for per, off in [(1, 0), (2, 1), (4, 0), (5, 3)]:
            got = api.ard_tile_bitmap_tdp(tn, tk, per, off).tolist()
            assert got == oprng.tile_bitmap_tdp(tn, tk, per, off)
        for p in (0.0, 0.3, 0.5, 1.0):
            got = api.ard_tile_bitmap_bernoulli(tn, tk, p, 8939, 2, 17).tolist()
            want = oprng.tile_bitmap_bernoulli(tn, tk, p, 8939, 2, 17)
            assert got == want
            assert api.ard_bitmap_popcount(np.array(got, np.uint32), tn * tk) == \
                opat.bitmap_popcount(want, tn * tk)


def test_list_free_row_plan_launches_nothing():
    """ard_plan_rows without a device list fills the host plan only, so it runs
    without a GPU."""
    for n, per, off in [(2048, 3, 1), (10, 16, 12), (7, 1, 0)]:
        plan = api.ard_plan_rows(n, per, off, None, stream=0)
        assert (plan.n, plan.period, plan.offset, plan.kept) == (n, per, off, opat.row_kept_count(n, per, off))
        assert not plan.d_idx
    with pytest.raises(api.ArdError):
        api.ard_plan_rows(10, 3, 3, None, stream=0)


def test_row_kept_matches_oracle():
    for n in range(0, 50):
        for per in range(1, 19):
            for off in range(per):
                assert api.ard_row_kept(n, per, off) == opat.row_kept_count(n, per, off)
    assert api.ard_row_kept(5, 0, 0) == -1
    assert api.ard_row_kept(5, 3, 3) == -1


@pytest.mark.parametrize("p", [0.3, 0.5, 0.7])
def test_search_plain_matches_closed_form(p):
    K, info = api.ard_search_distribution(p)
    Kstar = osearch.closed_form(p, 16)
    assert info.converged == 1 and info.iters < 100_000
    assert np.max(np.abs(K - Kstar)) < 2e-5
    assert abs(info.p_global - osearch.global_rate(K)) < 1e-14
    assert abs(info.p_global - p) < 0.01
    assert abs(K.sum() - 1.0) < 1e-12
    assert info.kkt_residual < 1e-5


@pytest.mark.parametrize("p,n", [(0.3, 16), (0.5, 16), (0.7, 16), (0.5, 256), (0.7, 2048)])
def test_search_mirror_matches_closed_form(p, n):
    o = api.ard_search_opts_default()
    o.mode = api.ARD_SEARCH_MIRROR
    o.n_max = n
    o.lr = 1.0
    K, info = api.ard_search_distribution(p, o)
    Kstar = osearch.closed_form(p, n)
    assert info.converged == 1
    assert np.max(np.abs(K - Kstar)) < 1e-7
    assert info.kkt_residual < 1e-6 and info.iters < 1000


def test_search_special_cases_and_errors():
    K, info = api.ard_search_distribution(0.0)
    assert K[0] == 1.0 and not K[1:].any() and info.iters == 0
    o = api.ard_search_opts_default()
    o.n_max = 1
    K, _ = api.ard_search_distribution(0.0, o)
    assert K.tolist() == [1.0]
    for bad_p in (15 / 16, 0.99, -0.1, float("nan")):
        with pytest.raises(api.ArdError) as e:
            api.ard_search_distribution(bad_p)
        assert e.value.status == _ffi.ARD_ERR_INVALID_ARG
        assert "rate" in e.value.message
    o = api.ard_search_opts_default()
    o.max_iters = 10
    with pytest.raises(api.ArdError) as e:
        api.ard_search_distribution(0.5, o)
    assert e.value.status == _ffi.ARD_ERR_NOT_CONVERGED
    assert abs(e.value.K.sum() - 1.0) < 1e-12 and e.value.info.iters == 10
    for field, val in (("lambda1", 1.0), ("lr", 0.0), ("n_max", 0), ("mode", 7), ("max_iters", 0)):
        o = api.ard_search_opts_default()
        setattr(o, field, val)
        with pytest.raises(api.ArdError) as e:
            api.ard_search_distribution(0.5, o)
        assert e.value.status == _ffi.ARD_ERR_INVALID_ARG


def test_sampler_argument_errors():
    K = np.array([0.5, 0.5])
    with pytest.raises(api.ArdError):
        api.ard_sample_row_pattern(np.zeros(3), 1, 0, 0)
    with pytest.raises(api.ArdError):
        api.ard_sample_row_pattern(np.array([0.5, -0.1]), 1, 0, 0)
    with pytest.raises(api.ArdError):
        api.ard_sample_row_pattern(K, 1, 1 << 24, 0)
    with pytest.raises(api.ArdError):
        api.ard_sample_row_pattern(K, 1, 0, 1 << 40)
    with pytest.raises(api.ArdError):
        api.ard_tile_bitmap_tdp(2, 2, 3, 3)
    with pytest.raises(api.ArdError):
        api.ard_tile_bitmap_bernoulli(2, 2, 1.5, 0, 0, 0)


def test_tile_call_validation_on_host():
    """Every tile-layer entry point rejects a bad descriptor, plan or operand
    on the host, before anything is launched (no GPU needed): each case below
    must fail validation, with the status its header states."""
    fake = 1 << 20  # 16-byte aligned, never dereferenced: every case fails before a launch

    def plan(**kw):
        p = dict(n=256, k=128, tile=64, tiles_n=4, tiles_k=2, nnz=3, d_bits=fake, d_row_ptr=fake,
                 d_row_cols=fake, d_col_ptr=fake, d_col_rows=fake, d_flat=fake, d_chunks=fake)
        p.update(kw)
        return _ffi.ard_tile_plan(**p)

    def desc(**kw):
        d = dict(dtype=api.ARD_BF16, batch=64, in_features=128, out_features=256, scale=1.0,
                 dropped=api.ARD_DROPPED_SKIP)
        d.update(kw)
        return _ffi.ard_tile_desc(**d)

    calls = {
        "fwd": lambda d, p, x=fake: api.ard_tile_fwd(d, p, x, fake, fake),
        "bwd_data": lambda d, p, x=fake: api.ard_tile_bwd_data(d, p, x, fake, fake),
        "bwd_weight": lambda d, p, x=fake: api.ard_tile_bwd_weight(d, p, x, fake, fake),
        "bwd": lambda d, p, x=fake: api.ard_tile_bwd(d, p, x, fake, fake, fake, fake),
    }
    bad = [
        (desc(dtype=7), plan(), _ffi.ARD_ERR_UNSUPPORTED, "dtype"),
        (desc(batch=0), plan(), _ffi.ARD_ERR_INVALID_ARG, "batch"),
        (desc(dropped=5), plan(), _ffi.ARD_ERR_INVALID_ARG, "dropped"),
        (desc(scale=float("nan")), plan(), _ffi.ARD_ERR_INVALID_ARG, "scale"),
        (desc(scale=float("inf")), plan(), _ffi.ARD_ERR_INVALID_ARG, "scale"),
        (desc(), plan(tile=48), _ffi.ARD_ERR_INVALID_ARG, "tile"),
        (desc(in_features=192), plan(), _ffi.ARD_ERR_INVALID_ARG, "does not match"),
        (desc(), plan(tiles_n=3), _ffi.ARD_ERR_INVALID_ARG, "grid"),
        (desc(), plan(nnz=9), _ffi.ARD_ERR_INVALID_ARG, "nnz"),
        (desc(), plan(nnz=-2), _ffi.ARD_ERR_INVALID_ARG, "nnz"),
        (desc(), plan(d_chunks=None), _ffi.ARD_ERR_INVALID_ARG, "NULL lists"),
    ]
    for name, call in calls.items():
        for d, p, status, msg in bad:
            with pytest.raises(api.ArdError) as e:
                call(d, p)
            assert e.value.status == status, (name, msg, e.value.message)
            assert msg in e.value.message, (name, msg, e.value.message)
        for x, msg in ((None, "is NULL"), (fake + 8, "aligned")):
            with pytest.raises(api.ArdError) as e:
                call(desc(), plan(), x)
            assert e.value.status == _ffi.ARD_ERR_INVALID_ARG and msg in e.value.message, (name, e.value.message)
        fn = getattr(_ffi.lib(), f"ard_tile_{name}")
        nargs = 6 if name == "bwd" else 4
        assert fn(None, ctypes.byref(plan()), *([None] * nargs)) == _ffi.ARD_ERR_INVALID_ARG  # NULL descriptor
        assert fn(ctypes.byref(desc()), None, *([None] * nargs)) == _ffi.ARD_ERR_INVALID_ARG  # NULL plan
