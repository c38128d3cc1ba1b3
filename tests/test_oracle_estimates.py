"""Pins of the oracle's point estimates and held-out fold-in (the step after the
sweep: the thesis's estimates after convergence and its perplexity).

* Normalisation: every theta row, every phi0 topic and every phig (group,
  topic) is a distribution over its outcomes.  The printed group estimate
  (base weighted by a T / (b + N)) fails this; the oracle's reading
  (b + a T) / (b + N) passes, and the next pin shows it is the Pitman-Yor
  predictive.
* Pitman-Yor predictive: for a restaurant with explicit tables, the
  probability that the next customer eats dish w, estimated by simulating the
  seating rule itself (join table j with weight n_j - a, open a new table with
  weight b + a T and draw its dish from the base), equals phig.
* Fold-in: the held-out Gibbs chain over a short test document, with phi
  fixed, leaves its states with the exact posterior p(z | w, phi, alpha) over
  all K^L topic vectors (enumerated).
* Perplexity closed form: with no training tokens, phi0 = phig = 1/V, so the
  held-out perplexity is V whatever the test documents and fold-in.
"""
import itertools
import math

import numpy as np
import pytest

import oracle
import synth


def _model(docs, K, V, alpha=0.5, a=0.5, b=2.0, gamma=0.5):
    words = np.array([w for _, d in docs for w in d], np.int32)
    doc_off = np.cumsum([0] + [len(d) for _, d in docs]).astype(np.int64)
    grp = np.array([g for g, _ in docs], np.int32)
    G = int(grp.max()) + 1 if len(docs) else 1
    return oracle.Model(words, doc_off, grp, G, K, V, alpha, a, b, gamma)


def test_estimates_are_distributions():
    cp = synth.generate(synth.workload(0), 2)
    m = oracle.Model(cp.words, cp.doc_off, cp.doc_group, cp.n_groups, 10, cp.vocab, 0.1, 0.5,
                     10.0, 0.01)
    z, r, c = m.initial_state(4)
    for sw in range(3):
        m.sweep(c, z, r, sw, 9)
    theta, phi0, phig = m.estimates(z, c)
    np.testing.assert_allclose(theta.sum(1), 1.0, rtol=1e-13)
    np.testing.assert_allclose(phi0.sum(1), 1.0, rtol=1e-13)
    np.testing.assert_allclose(phig.sum(2), 1.0, rtol=1e-13)
    assert theta.min() > 0 and phi0.min() > 0 and phig.min() > 0
    # the printed weight a T / (b + N) would leave each phig row summing to N / (b + N)
    N = c.Ngk.astype(np.float64)
    printed = phig.sum(2) - (m.b / (m.b + N))
    assert np.all(np.abs(printed - N / (m.b + N)) < 1e-12)


@pytest.mark.parametrize("a,b", [(0.5, 2.0), (0.0, 3.0), (0.8, 0.7)])
def test_group_estimate_is_the_pitman_yor_predictive(a, b):
    # one group, one topic: tables with explicit sizes per dish
    tables = {0: [3, 1], 1: [2], 2: [1, 1, 1], 4: [5]}  # dish -> customers per table
    V, K = 6, 1
    words, rr = [], []
    for w, sizes in tables.items():
        for sz in sizes:
            words += [w] * sz
            rr += [1] + [0] * (sz - 1)
    m = _model([(0, words)], K, V, alpha=1.0, a=a, b=b, gamma=0.3)
    z = np.zeros(len(words), np.int32)
    r = np.array(rr, np.uint8)
    c = m.rebuild(z, r)
    _, phi0, phig = m.estimates(z, c)
    # simulate the seating rule of the next customer
    rng = np.random.default_rng(11)
    sizes = [(w, s) for w, ss in tables.items() for s in ss]
    T, N = len(sizes), sum(s for _, s in sizes)
    weights = np.array([s - a for _, s in sizes] + [b + a * T]) / (b + N)
    draws = 2_000_000
    pick = rng.choice(len(weights), size=draws, p=weights)
    dish = np.empty(draws, np.int64)
    old = pick < T
    dish[old] = np.array([w for w, _ in sizes])[pick[old]]
    dish[~old] = rng.choice(V, size=int((~old).sum()), p=phi0[0])
    freq = np.bincount(dish, minlength=V) / draws
    se = np.sqrt(phig[0, 0] * (1 - phig[0, 0]) / draws)
    assert np.all(np.abs(freq - phig[0, 0]) < 6 * se + 1e-12), (freq, phig[0, 0])


FOLDIN_CASES = [
    # (training docs, K, V, hypers, test document words)
    ([(0, [0, 1, 0, 2]), (0, [1, 1, 2])], 2, 3, dict(alpha=0.5, a=0.5, b=2.0, gamma=0.5), [0, 1, 2]),
    ([(0, [0, 0, 0, 1]), (1, [1, 2, 2])], 3, 3, dict(alpha=0.2, a=0.0, b=1.0, gamma=0.2), [2, 0]),
]


@pytest.mark.parametrize("case", range(len(FOLDIN_CASES)))
def test_foldin_chain_matches_exact_posterior(case):
    docs, K, V, hyp, test = FOLDIN_CASES[case]
    m = _model(docs, K, V, **hyp)
    z, r, c = m.initial_state(3)
    for sw in range(4):
        m.sweep(c, z, r, sw, 5)
    _, _, phig = m.estimates(z, c)
    g = 0
    L = len(test)
    # exact posterior over z in [K]^L: prod_n phig[g, z_n, w_n] * DirMult(c(z) | alpha)
    post = np.zeros(K ** L)
    for code, zz in enumerate(itertools.product(range(K), repeat=L)):
        cnt = np.bincount(np.array(zz), minlength=K)
        lp = sum(math.log(phig[g, zz[n], test[n]]) for n in range(L))
        lp += sum(math.lgamma(cnt[k] + m.alpha) - math.lgamma(m.alpha) for k in range(K))
        post[code] = math.exp(lp)
    post /= post.sum()
    # final states of many independent fold-in chains (one test document each)
    runs, sweeps = 20000, 12
    words = np.array(test * runs, np.int32)
    off = (np.arange(runs + 1) * L).astype(np.int64)
    grp = np.full(runs, g, np.int32)
    _, zt, _ = m.heldout(phig, words, off, grp, sweeps, 77)
    codes = np.zeros(runs, np.int64)
    for n in range(L):
        codes = codes * K + zt[n::L]
    freq = np.bincount(codes, minlength=K ** L) / runs
    tv = 0.5 * np.abs(freq - post).sum()
    assert tv < 0.03, (tv, freq, post)


def test_perplexity_is_vocabulary_size_without_training_tokens():
    V, K = 9, 4
    m = _model([(0, []), (1, [])], K, V, alpha=0.3, a=0.4, b=5.0, gamma=0.2)
    z = np.zeros(0, np.int32)
    r = np.zeros(0, np.uint8)
    c = m.rebuild(z, r)
    _, phi0, phig = m.estimates(z, c)
    np.testing.assert_allclose(phig, 1.0 / V, rtol=1e-15)
    rng = np.random.default_rng(5)
    lens = [0, 1, 7, 30]
    words = rng.integers(0, V, size=sum(lens)).astype(np.int32)
    off = np.cumsum([0] + lens).astype(np.int64)
    grp = np.array([0, 1, 1, 0], np.int32)
    total, _, ll = m.heldout(phig, words, off, grp, 5, 3)
    assert ll[0] == 0.0
    ppl = math.exp(-total / sum(lens))
    assert abs(ppl - V) < 1e-12 * V
