"""Pins of the oracle's generalised Stirling table S^n_{t,a}.

The table is the oracle's fp64 evaluation of the recurrence stated with the
PYP joint (thesis, Corollary 17 passage of the SPDP chapter).  None of the
checks below re-runs that recurrence: each one is a fact the numbers must obey
by other mathematics.
"""
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle


def logS(table, n, t):
    return table[oracle.tri(n, t)]


@pytest.mark.parametrize("a", [0.0, 0.3, 0.5, 0.8])
def test_closed_forms(a):
    nmax = 60
    T = oracle.stirling_log_table(nmax, a)
    for n in range(0, nmax + 1):
        # S^n_n = 1
        assert logS(T, n, n) == pytest.approx(0.0, abs=1e-12)
        # S^n_0 = delta_{n,0}
        if n > 0:
            assert logS(T, n, 0) == -math.inf
    for n in range(1, nmax + 1):
        # S^n_1 = prod_{j=1}^{n-1} (j - a)  (a single table seating everyone)
        want = sum(math.log(j - a) for j in range(1, n))
        assert logS(T, n, 1) == pytest.approx(want, rel=1e-12, abs=1e-12)
    for n in range(2, nmax + 1):
        # S^n_{n-1} = C(n, 2) (1 - a)
        want = math.log(math.comb(n, 2) * (1 - a))
        assert logS(T, n, n - 1) == pytest.approx(want, rel=1e-12, abs=1e-12)


def test_a_zero_is_unsigned_stirling_first_kind():
    # Coefficients of the rising factorial x (x+1) ... (x+n-1) are the unsigned
    # Stirling numbers of the first kind; build them by polynomial products.
    nmax = 40
    T = oracle.stirling_log_table(nmax, 0.0)
    poly = [1]  # n = 0
    for n in range(1, nmax + 1):
        # multiply by (x + n - 1)
        new = [0] * (len(poly) + 1)
        for i, c in enumerate(poly):
            new[i + 1] += c
            new[i] += c * (n - 1)
        poly = new
        for t in range(1, n + 1):
            assert math.exp(logS(T, n, t) - math.log(poly[t])) == pytest.approx(1.0, rel=1e-11)
        assert sum(poly) == math.factorial(n)


def _log_poch(x, y, T):
    return sum(math.log(x + j * y) for j in range(T))


@pytest.mark.parametrize("a,b", [(0.5, 10.0), (0.8, 100.0), (0.7, 50.0), (0.0, 3.0), (0.2, 0.5)])
def test_pyp_normalisation(a, b):
    # The PYP table-count distribution p(T = t | n) = (b|a)_t S^n_{t,a} / (b)_n sums
    # to one for every b: a polynomial identity in b that fixes all S^n_t.
    nmax = 200
    T = oracle.stirling_log_table(nmax, a)
    for n in (1, 2, 3, 7, 20, 64, 137, 200):
        terms = np.array([_log_poch(b, a, t) + logS(T, n, t) for t in range(1, n + 1)])
        m = terms.max()
        log_sum = m + math.log(np.exp(terms - m).sum())
        assert log_sum == pytest.approx(_log_poch(b, 1.0, n), rel=1e-12)


def test_normalisation_exact_rationals():
    # The same identity with the Pochhammer symbols in exact rationals, so the
    # only rounding is that of the table entries themselves.
    a, b = Fraction(1, 2), Fraction(3)
    nmax = 12
    T = oracle.stirling_log_table(nmax, float(a))
    for n in range(1, nmax + 1):
        lhs = Fraction(0)
        for t in range(1, n + 1):
            poch = Fraction(1)
            for j in range(t):
                poch *= b + j * a
            lhs += poch * Fraction(math.exp(logS(T, n, t)))
        rhs = Fraction(1)
        for j in range(n):
            rhs *= b + j
        assert float(lhs / rhs) == pytest.approx(1.0, rel=1e-13)


@pytest.mark.parametrize("a,b", [(0.5, 10.0), (0.8, 100.0)])
def test_expected_tables(a, b):
    # E[T_n] = (b/a) [ (b+a)_n / (b)_n - 1 ]  for the two-parameter PYP.
    nmax = 300
    T = oracle.stirling_log_table(nmax, a)
    for n in (1, 5, 50, 300):
        logp = np.array([_log_poch(b, a, t) + logS(T, n, t) - _log_poch(b, 1.0, n)
                         for t in range(1, n + 1)])
        mean = float((np.arange(1, n + 1) * np.exp(logp)).sum())
        want = (b / a) * (math.exp(_log_poch(b + a, 1.0, n) - _log_poch(b, 1.0, n)) - 1.0)
        assert mean == pytest.approx(want, rel=1e-11)


def test_large_n_normalisation():
    # The table at the row counts the largest workload needs (a few thousand).
    a, b = 0.8, 100.0
    nmax = 6000
    T = oracle.stirling_log_table(nmax, a)
    # cumulative log (b|a)_t for t = 0..nmax
    cum = np.concatenate([[0.0], np.cumsum(np.log(b + a * np.arange(nmax)))])
    for n in (1000, 4321, 6000):
        terms = cum[1:n + 1].copy()
        row = T[oracle.tri(n, 1): oracle.tri(n, n) + 1]
        terms = terms + row
        m = terms.max()
        log_sum = m + math.log(np.exp(terms - m).sum())
        assert log_sum == pytest.approx(_log_poch(b, 1.0, n), rel=1e-12)
