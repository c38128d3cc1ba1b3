"""Pins of the oracle's topic-model comparison (Hellinger distance and topic
alignment), none of which re-types its formula:

* Closed forms from the Bhattacharyya coefficient BC = 1 - H^2 of known
  families: two geometric laws, BC = sqrt((1-x)(1-y)) / (1 - sqrt(xy)), and
  two binomial laws Bin(n, x), Bin(n, y), BC = (sqrt(xy) + sqrt((1-x)(1-y)))^n
  (a sum over outcomes collapsed by the geometric series / binomial theorem).
* Special cases: identical laws are at distance 0, laws with disjoint
  supports at 1.
* Metric and bounds: symmetry, triangle inequality, and H^2 <= TV <= sqrt(2) H
  between Hellinger and total-variation distance, on random laws.
* Alignment: the matching of least total distance equals brute force over
  every permutation (square) and every injection (rectangular); a planted
  permutation of the same topics is recovered with total 0.
"""
import itertools
import math

import numpy as np
import pytest
from scipy.stats import binom

import oracle


@pytest.mark.parametrize("x,y", [(0.2, 0.5), (0.05, 0.3), (0.4, 0.4), (0.6, 0.1)])
def test_geometric_closed_form(x, y):
    V = 400  # tails below 1e-80
    n = np.arange(V)
    p = (1 - x) * x ** n
    q = (1 - y) * y ** n
    H = oracle.hellinger(p[None], q[None])[0, 0]
    bc = math.sqrt((1 - x) * (1 - y)) / (1 - math.sqrt(x * y))
    assert abs(H * H - (1 - bc)) < 1e-14


@pytest.mark.parametrize("n,x,y", [(10, 0.3, 0.6), (50, 0.5, 0.52), (200, 0.1, 0.9)])
def test_binomial_closed_form(n, x, y):
    k = np.arange(n + 1)
    P = binom.pmf(k, n, x)[None]
    Q = binom.pmf(k, n, y)[None]
    H = oracle.hellinger(P, Q)[0, 0]
    bc = (math.sqrt(x * y) + math.sqrt((1 - x) * (1 - y))) ** n
    assert abs(H * H - (1 - bc)) < 1e-13


def test_identical_and_disjoint():
    rng = np.random.default_rng(0)
    P = rng.dirichlet(np.full(30, 0.3), size=4)
    assert np.all(np.diag(oracle.hellinger(P, P)) == 0.0)
    A = np.zeros((2, 6))
    A[0, :3] = [0.2, 0.3, 0.5]
    A[1, 3:] = [0.6, 0.3, 0.1]
    H = oracle.hellinger(A, A[::-1])
    assert abs(H[0, 0] - 1.0) < 1e-15 and abs(H[1, 1] - 1.0) < 1e-15
    assert H[0, 1] == 0.0 and H[1, 0] == 0.0


def test_metric_and_total_variation_bounds():
    rng = np.random.default_rng(1)
    P = rng.dirichlet(np.full(50, 0.2), size=12)
    Q = rng.dirichlet(np.full(50, 0.5), size=7)
    H = oracle.hellinger(P, Q)
    assert H.shape == (12, 7)
    np.testing.assert_allclose(oracle.hellinger(Q, P), H.T, rtol=0, atol=1e-15)
    HP = oracle.hellinger(P, P)
    for i, j in itertools.product(range(12), repeat=2):
        assert np.all(HP[i, j] <= H[i] + H[j] + 1e-15)
    tv = 0.5 * np.abs(P[:, None, :] - Q[None, :, :]).sum(-1)
    assert np.all(H * H <= tv + 1e-15)
    assert np.all(tv <= math.sqrt(2) * H + 1e-15)


@pytest.mark.parametrize("kp,kq", [(5, 5), (6, 6), (3, 5), (1, 4)])
def test_alignment_is_least_total_distance(kp, kq):
    rng = np.random.default_rng(kp * 10 + kq)
    H = rng.random((kp, kq))
    match, total = oracle.align_topics(H)
    assert len(set(match.tolist())) == kp and match.min() >= 0 and match.max() < kq
    assert abs(H[np.arange(kp), match].sum() - total) < 1e-12
    best = min(sum(H[i, c[i]] for i in range(kp))
               for c in itertools.permutations(range(kq), kp))
    assert abs(total - best) < 1e-12


def test_alignment_recovers_a_planted_permutation():
    rng = np.random.default_rng(7)
    P = rng.dirichlet(np.full(200, 0.1), size=9)
    perm = rng.permutation(9)
    Q = P[perm]  # topic j of Q is topic perm[j] of P
    match, total = oracle.align_topics(oracle.hellinger(P, Q))
    assert total == 0.0
    np.testing.assert_array_equal(perm[match], np.arange(9))
