"""Pins of the oracle's look-ahead memory estimate (Algorithm 1), CPU only.

Fixed against brute-force enumeration of the accept/reject process the algorithm's terms count
(an acceptance costs one iteration, a rejection pp), scipy's binomial pmf, the binomial theorem
(pp = 1), the closed forms at theta = 1 and theta = 0, additivity over requests, and precision 0.
"""
import itertools

import numpy as np
import pytest
from scipy.stats import binom

import oracle


def brute(i, pp, theta, tau):
    """(E_gen, P[generated >= tau]) over every accept/reject string costing exactly i iterations."""
    gen = fin = 0.0
    for n_rej in range(i // pp + 1):
        n_acc = i - pp * n_rej
        for pos in itertools.combinations(range(n_acc + n_rej), n_rej):   # every ordering
            prob = theta ** n_acc * (1 - theta) ** n_rej
            k = n_acc + n_rej
            gen += k * prob
            fin += prob if k >= tau else 0.0
    return gen, fin


@pytest.mark.parametrize("pp", [2, 3, 4])
@pytest.mark.parametrize("theta", [0.0, 0.35, 0.8, 1.0])
def test_brute_force_enumeration(pp, theta):
    iters = 14
    for tau in (1, 3, 6, 9, 14, 20):
        mem, e_gen, e_nfin, e_lfin = oracle.lookahead([0], [tau], [1.0], pp, theta, iters)
        for i in range(1, iters + 1):
            g, f = brute(i, pp, theta, tau)
            assert e_gen[i - 1] == pytest.approx(g, rel=1e-12, abs=1e-15)
            assert e_nfin[i - 1] == pytest.approx(f, rel=1e-12, abs=1e-15)
            assert mem[i - 1] == pytest.approx((1 - f) * g, rel=1e-12, abs=1e-12)


@pytest.mark.parametrize("pp", [1, 2, 4, 7])
@pytest.mark.parametrize("theta", [0.05, 0.5, 0.93])
def test_expected_generation_matches_scipy_binomial(pp, theta):
    _, e_gen, _, _ = oracle.lookahead([], [], [], pp, theta, 64)
    for i in range(1, 65):
        ref = sum((i - (pp - 1) * w) * binom.pmf(i - pp * w, i - (pp - 1) * w, theta) for w in range(i // pp + 1))
        assert e_gen[i - 1] == pytest.approx(ref, rel=1e-10)


def test_depth_one_is_the_binomial_theorem():
    rng = np.random.default_rng(1)
    n = 50
    ell = rng.integers(1, 5000, n)
    tau = rng.integers(1, 80, n)
    prec = rng.uniform(0.5, 1.0, n)
    mem, e_gen, e_nfin, _ = oracle.lookahead(ell, tau, prec, 1, 0.6, 64)
    i = np.arange(1, 65)
    np.testing.assert_allclose(e_gen, i, rtol=1e-12)     # k = i for every w, sum_w p = 1
    nfin = np.array([(prec * (tau <= j)).sum() for j in i])
    np.testing.assert_allclose(e_nfin, nfin, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("pp", [1, 2, 3, 5])
def test_theta_one_closed_form(pp):
    # every speculation accepted: k = i exactly, requests with tau <= i finish
    rng = np.random.default_rng(2)
    n = 40
    ell = rng.integers(0, 10000, n)
    tau = rng.integers(1, 70, n)
    mem, e_gen, e_nfin, e_lfin = oracle.lookahead(ell, tau, np.ones(n), pp, 1.0, 64)
    for i in range(1, 65):
        done = tau <= i
        assert e_gen[i - 1] == i
        assert e_nfin[i - 1] == done.sum()
        assert mem[i - 1] == ell.sum() + (n - done.sum()) * i - ell[done].sum()


@pytest.mark.parametrize("pp", [2, 3, 4])
def test_theta_zero_closed_form(pp):
    # every speculation rejected: the process lands on i only when pp divides it, with k = i / pp
    tau = np.array([1, 2, 5, 8, 16, 30])
    ell = np.array([100, 200, 300, 400, 500, 600])
    prec = np.array([0.9, 0.8, 0.7, 0.6, 0.5, 0.4])
    mem, e_gen, e_nfin, e_lfin = oracle.lookahead(ell, tau, prec, pp, 0.0, 64)
    for i in range(1, 65):
        hit = i % pp == 0
        k = i // pp
        assert e_gen[i - 1] == (k if hit else 0)
        fin = prec * ((tau <= k) & hit)
        assert e_nfin[i - 1] == pytest.approx(fin.sum(), abs=1e-15)
        assert e_lfin[i - 1] == pytest.approx((ell * fin).sum(), abs=1e-12)


def test_additive_over_requests_and_zero_precision():
    rng = np.random.default_rng(3)
    n = 30
    ell = rng.integers(1, 8000, n)
    tau = rng.integers(1, 65, n)
    prec = rng.uniform(0, 1, n)
    full = oracle.lookahead(ell, tau, prec, 3, 0.7, 64)[0]
    a = oracle.lookahead(ell[:12], tau[:12], prec[:12], 3, 0.7, 64)[0]
    b = oracle.lookahead(ell[12:], tau[12:], prec[12:], 3, 0.7, 64)[0]
    np.testing.assert_allclose(full, a + b, rtol=1e-12)
    mem, e_gen, e_nfin, e_lfin = oracle.lookahead(ell, tau, np.zeros(n), 3, 0.7, 64)
    assert (e_nfin == 0).all() and (e_lfin == 0).all()
    np.testing.assert_allclose(mem, ell.sum() + n * e_gen, rtol=1e-14)


def test_no_requests_and_bad_arguments():
    mem = oracle.lookahead([], [], [], 2, 0.5, 64)[0]
    assert (mem == 0).all()
    for pp, theta, iters in ((0, 0.5, 64), (2, 1.5, 64), (2, -0.1, 64), (2, float("nan"), 64), (2, 0.5, 0)):
        with pytest.raises(ValueError):
            oracle.lookahead([5], [3], [1.0], pp, theta, iters)
