"""Pins of the oracle's Alg. 1 (Sec. III-C) and Eq. 3."""
import json
import os

import numpy as np
import pytest
from scipy.optimize import minimize

from oracle import search

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
EX = json.load(open(os.path.join(GOLDEN, "paper_examples.json")))


def test_drop_rates_vector_of_alg1():
    ex = EX["drop_rates_p_u"]
    want = np.array(ex["numerators"], float) / np.array(ex["denominators"], float)
    assert np.array_equal(search.drop_rates(ex["N"]), want)


@pytest.mark.parametrize("p", [0.3, 0.5, 0.7])
def test_closed_form_matches_a_generic_constrained_solver(p):
    n, lam1 = 8, 0.9
    K = search.closed_form(p, n, lam1)
    cons = ({"type": "eq", "fun": lambda d: d.sum() - 1.0},)
    res = minimize(lambda d: search.loss(np.clip(d, 1e-300, 1), p, lam1, 1 - lam1),
                   np.full(n, 1.0 / n), method="SLSQP", constraints=cons,
                   bounds=[(1e-12, 1.0)] * n, options={"ftol": 1e-16, "maxiter": 2000})
    assert res.success
    assert np.max(np.abs(res.x - K)) < 2e-4
    assert search.loss(K, p, lam1, 1 - lam1) <= search.loss(res.x, p, lam1, 1 - lam1) + 1e-12


@pytest.mark.parametrize("p", [0.3, 0.5, 0.7])
def test_paper_iteration_converges_to_the_closed_form(p):
    K = search.closed_form(p, 16)
    d, iters, ok = search.search_gd(p, 16)
    assert ok and iters < 100_000
    assert np.max(np.abs(d - K)) < 2e-5


@pytest.mark.parametrize("p", [0.3, 0.5, 0.7])
def test_global_rate_close_to_target(p):
    K = search.closed_form(p, 16)
    assert abs(K.sum() - 1.0) < 1e-12
    assert abs(search.global_rate(K) - p) < 0.01
    assert search.kkt_residual(K, p, 0.99) < 1e-12


def test_kkt_residual_detects_non_optimum():
    K = search.closed_form(0.5, 16)
    K2 = K.copy()
    K2[0] += 0.01
    K2[5] -= 0.01
    assert search.kkt_residual(K2, 0.5, 0.99) > 1e-4


def test_special_cases():
    assert np.array_equal(search.closed_form(0.3, 1), np.ones(1))
    e = search.distribution_for_rate(0.0, 16)
    assert e[0] == 1.0 and e[1:].sum() == 0.0
    with pytest.raises(ValueError):
        search.distribution_for_rate(15 / 16, 16)
    with pytest.raises(ValueError):
        search.distribution_for_rate(-0.1, 16)
    # as the entropy weight vanishes the expected rate reaches p
    K = search.closed_form(0.5, 16, lam1=1 - 1e-7)
    assert abs(search.global_rate(K) - 0.5) < 1e-5
    # with lambda1 -> 0 only entropy remains: the uniform distribution
    K = search.closed_form(0.5, 16, lam1=1e-9)
    assert np.max(np.abs(K - 1 / 16)) < 1e-6


def test_gibbs_form_is_stationary():
    p, n, lam1 = 0.6, 12, 0.95
    K = search.closed_form(p, n, lam1)
    # log-odds against p_u are linear: log k_i - log k_1 = beta * p_u[i]
    pu = search.drop_rates(n)
    beta = (np.log(K[1:]) - np.log(K[0])) / pu[1:]
    assert np.max(np.abs(beta - beta.mean())) < 1e-8
