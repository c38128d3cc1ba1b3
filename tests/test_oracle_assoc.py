"""Pins of the oracle with word associations (non-identity transformation
matrices P^g):

* Reduction: with P^g = I (one source per row, the word itself, p = 1) every
  association routine gives exactly the P = I oracle's result (initial state,
  weights, snapshot and sequential sweeps, joint, estimates).
* Generative process: the association joint log p(W, Z, V, R), summed over
  every head labelling R and every source choice of every head, equals
  p(W, Z) from brute-force enumeration of the Chinese-restaurant seatings in
  which each new table draws its source from the shadow base's Polya urn and
  then its word from column v of P^g (tests/brute.py).
* Conditionals: the K (S + 1) weights of a token are ratios of that joint,
  including exact zeros; the only head of a cell that keeps other customers
  stays its head but may change its source.
* Chain: the sequential chain's state frequencies match the exact posterior
  over every (z, r, source) state.
* Estimates: with column-stochastic P^g the group estimate is a distribution
  over words.
"""
import itertools
import math

import numpy as np
import pytest

import oracle
import synth
from tests import brute


def _corpus(docs):
    words = np.array([w for _, d in docs for w in d], np.int32)
    off = np.cumsum([0] + [len(d) for _, d in docs]).astype(np.int64)
    grp = np.array([g for g, _ in docs], np.int32)
    return words, off, grp


def _identity(G, V):
    return (np.arange(G * V + 1, dtype=np.int64), np.tile(np.arange(V, dtype=np.int32), G),
            np.ones(G * V))


def _assoc_dict(row_off, src, p, G, V):
    out = {}
    for q in range(G * V):
        g, w = divmod(q, V)
        out[(g, w)] = {int(src[e]): float(p[e]) for e in range(row_off[q], row_off[q + 1])}
    return out


HYP = dict(alpha=0.3, a=0.5, b=2.0, gamma=0.4)


def test_identity_associations_reduce_to_the_plain_model():
    cp = synth.generate(synth.workload(0), 3)
    wl = synth.workload(0)
    args = (cp.words, cp.doc_off, cp.doc_group, cp.n_groups, wl.K, cp.vocab, wl.alpha, wl.a,
            wl.b, wl.gamma)
    m = oracle.Model(*args)
    ma = oracle.AssocModel(*args, *_identity(cp.n_groups, cp.vocab))
    assert ma.S == 1
    z, r, c = m.initial_state(5)
    za, ra, sa, ca = ma.initial_state(5)
    np.testing.assert_array_equal(z, za)
    np.testing.assert_array_equal(r, ra)
    assert not sa.any()
    for f in ("n", "t", "Ngk", "Tgk", "Bkw", "Bk"):
        np.testing.assert_array_equal(getattr(c, f), getattr(ca, f))
    # weights of the first document's tokens
    d0, d1 = cp.doc_off[0], cp.doc_off[1]
    crow = np.bincount(z[d0:d1], minlength=wl.K)
    for i in range(d0, d1):
        w = m.token_weights(c, crow, cp.doc_group[0], cp.words[i], z[i], r[i])
        wa = ma.token_weights(ca, crow, cp.doc_group[0], cp.words[i], za[i], ra[i], sa[i])
        if w is None:
            # the sole head keeps its cell; with one source its only outcome
            # is its current state
            assert np.flatnonzero(wa).tolist() == [2 * z[i]]
        else:
            np.testing.assert_array_equal(w, wa)
    for sw in range(3):
        assert m.sweep(c, z, r, sw, 9) == ma.sweep(ca, za, ra, sa, sw, 9)
    for sw in range(3, 5):
        m.sweep(c, z, r, sw, 9, mode="sequential")
        ma.sweep(ca, za, ra, sa, sw, 9, mode="sequential")
    np.testing.assert_array_equal(z, za)
    np.testing.assert_array_equal(r, ra)
    assert not sa.any()
    assert m.loglik(z, r, c) == ma.loglik(za, ra, sa, ca)
    for x, y in zip(m.estimates(z, c), ma.estimates(za, ca)):
        np.testing.assert_array_equal(x, y)


ASSOC_CASES = [
    # docs, K, V, P (per group: {w: {v: p}}) -- columns sum to one
    ([(0, [0, 1, 0]), (0, [0, 1]), (1, [2, 0]), (1, [0, 2])], 2, 3,
     [{0: {0: 0.7, 1: 0.3}, 1: {1: 0.7, 0: 0.3}, 2: {2: 1.0}},
      {0: {0: 0.6, 2: 0.4}, 1: {1: 1.0}, 2: {2: 0.6, 0: 0.4}}]),
    ([(0, [0, 0, 1]), (1, [1, 2]), (1, [2, 2, 0])], 2, 3,
     [{0: {0: 0.5, 2: 0.5}, 1: {1: 1.0}, 2: {2: 0.5, 0: 0.5}},
      {0: {0: 0.8, 1: 0.1, 2: 0.1}, 1: {1: 0.8, 2: 0.1, 0: 0.1}, 2: {2: 0.8, 0: 0.1, 1: 0.1}}]),
]


def _assoc_model(case, K=None, hyp=HYP):
    docs, K0, V, P = ASSOC_CASES[case]
    words, off, grp = _corpus(docs)
    G = int(grp.max()) + 1
    row_off, src, p = [0], [], []
    for g in range(G):
        for w in range(V):
            for v, pv in P[g][w].items():
                src.append(v)
                p.append(pv)
            row_off.append(len(src))
    return oracle.AssocModel(words, off, grp, G, K or K0, V, **hyp, row_off=row_off, src=src,
                             p=p)


def _nsrc(m, i):
    """Length of the source list of token i's row (g, w)."""
    g = int(m.doc_group[np.searchsorted(m.doc_off, i, "right") - 1])
    q = g * m.V + int(m.words[i])
    return int(m.row_off[q + 1] - m.row_off[q])


def _labellings(m, z):
    """Every (r, s) over the tokens: a head takes any slot of its source list."""
    per_tok = [[(0, 0)] + [(1, sl) for sl in range(_nsrc(m, i))] for i in range(m.N)]
    for combo in itertools.product(*per_tok):
        yield (np.array([x[0] for x in combo], np.uint8),
               np.array([x[1] for x in combo], np.uint8))


@pytest.mark.parametrize("case", range(len(ASSOC_CASES)))
def test_joint_summed_over_labellings_and_sources_equals_crp_marginal(case):
    m = _assoc_model(case)
    assoc = _assoc_dict(m.row_off, m.src, m.p, m.G, m.V)
    rng = np.random.default_rng(case)
    for _ in range(3):
        z = rng.integers(0, m.K, size=m.N).astype(np.int32)
        acc = []
        for r, s in _labellings(m, z):
            c = m.rebuild(z, r, s)
            ll = m.loglik(z, r, s, c)
            if ll != -math.inf:
                acc.append(ll)
        acc = np.array(acc)
        mx = acc.max()
        log_sum = mx + math.log(np.exp(acc - mx).sum())
        want = brute.log_p_Z(list(m.doc_off), list(z), m.K, m.alpha) + math.log(
            brute.p_W_given_Z_assoc(list(m.words), list(m.doc_off), list(m.doc_group), list(z),
                                    m.G, m.K, m.V, m.a, m.b, m.gamma, assoc))
        assert log_sum == pytest.approx(want, rel=1e-12, abs=1e-12)


@pytest.mark.parametrize("case", range(len(ASSOC_CASES)))
@pytest.mark.parametrize("K", [1, 2, 3])
def test_conditionals_are_joint_ratios(case, K):
    m = _assoc_model(case, K)
    S1 = m.S + 1
    rng = np.random.default_rng(31 + K + 7 * case)
    checked = 0
    for _ in range(8):
        z = rng.integers(0, K, size=m.N).astype(np.int32)
        r = rng.integers(0, 2, size=m.N).astype(np.uint8)
        s = np.zeros(m.N, np.uint8)
        for i in range(m.N):
            s[i] = rng.integers(0, _nsrc(m, i)) if r[i] else 0
        c = m.rebuild(z, r, s)
        m.repair(z, r, s, c)
        assert math.isfinite(m.loglik(z, r, s, c))
        for d in range(m.D):
            g = int(m.doc_group[d])
            crow = np.bincount(z[m.doc_off[d]:m.doc_off[d + 1]], minlength=K)
            for i in range(m.doc_off[d], m.doc_off[d + 1]):
                w = m.token_weights(c, crow, g, m.words[i], z[i], r[i], s[i])
                lls = np.full(K * S1, -math.inf)
                nsrc = _nsrc(m, i)
                for j in range(K * S1):
                    k, sl = divmod(j, S1)
                    if sl < m.S and sl >= nsrc:
                        continue  # an empty slot of a shorter source list
                    z2, r2, s2 = z.copy(), r.copy(), s.copy()
                    z2[i] = k
                    r2[i] = 1 if sl < m.S else 0
                    s2[i] = sl if sl < m.S else 0
                    lls[j] = m.loglik(z2, r2, s2, m.rebuild(z2, r2, s2))
                assert w is not None
                fin = np.isfinite(lls)
                assert np.array_equal(w > 0, fin), (w, lls)
                pj = np.zeros(K * S1)
                pj[fin] = np.exp(lls[fin] - lls[fin].max())
                pj /= pj.sum()
                np.testing.assert_allclose(w / w.sum(), pj, rtol=1e-10, atol=1e-14)
                checked += 1
    assert checked > 20


def _enumerate_posterior(m):
    S1 = m.S + 1
    base = m.K * S1
    nb = base ** m.N
    lp = np.full(nb, -math.inf)
    for code in range(nb):
        z = np.empty(m.N, np.int32)
        r = np.empty(m.N, np.uint8)
        s = np.empty(m.N, np.uint8)
        x = code
        ok = True
        for i in range(m.N):
            dgt = x % base
            x //= base
            z[i], sl = divmod(dgt, S1)
            r[i] = 1 if sl < m.S else 0
            s[i] = sl if sl < m.S else 0
            if r[i] and s[i] >= _nsrc(m, i):
                ok = False
        if ok:
            lp[code] = m.loglik(z, r, s, m.rebuild(z, r, s))
    fin = np.isfinite(lp)
    out = np.zeros(nb)
    out[fin] = np.exp(lp[fin] - lp[fin].max())
    return out / out.sum()


def test_sequential_chain_matches_exact_posterior():
    docs = [(0, [0, 1, 0]), (1, [0, 2])]
    words, off, grp = _corpus(docs)
    P = [{0: {0: 0.7, 1: 0.3}, 1: {1: 0.7, 0: 0.3}, 2: {2: 1.0}},
         {0: {0: 0.6, 2: 0.4}, 1: {1: 1.0}, 2: {2: 0.6, 0: 0.4}}]
    row_off, src, p = [0], [], []
    for g in range(2):
        for w in range(3):
            for v, pv in P[g][w].items():
                src.append(v)
                p.append(pv)
            row_off.append(len(src))
    m = oracle.AssocModel(words, off, grp, 2, 2, 3, alpha=0.5, a=0.4, b=1.5, gamma=0.5,
                          row_off=row_off, src=src, p=p)
    post = _enumerate_posterior(m)
    z, r, s, c = m.initial_state(2)
    m.chain_histogram(c, z, r, s, 0, 10_000, seed=5)
    hist = m.chain_histogram(c, z, r, s, 10_000, 4_000_000, seed=5)
    freq = hist / hist.sum()
    tv = 0.5 * np.abs(freq - post).sum()
    assert tv < 0.01, tv
    assert np.all(post[hist > 0] > 0)
    big = post > 0.01
    np.testing.assert_allclose(freq[big], post[big], rtol=0.06)


def test_group_estimate_is_a_distribution_with_associations():
    cp = synth.generate(synth.workload(0), 1)
    wl = synth.workload(0)
    ro, src, p = synth.associations(cp.n_groups, cp.vocab, 4, 0.3, 2)
    m = oracle.AssocModel(cp.words, cp.doc_off, cp.doc_group, cp.n_groups, wl.K, cp.vocab,
                          wl.alpha, wl.a, wl.b, wl.gamma, ro, src, p)
    z, r, s, c = m.initial_state(1)
    for sw in range(2):
        m.sweep(c, z, r, s, sw, 4)
    theta, phi0, phig = m.estimates(z, c)
    np.testing.assert_allclose(phi0.sum(1), 1.0, rtol=1e-13)
    np.testing.assert_allclose(phig.sum(2), 1.0, rtol=1e-12)
    assert phig.min() > 0
    # heads carry sources: the base counts are keyed by source, and sum to T
    assert c.Bk.sum() == c.Tgk.sum() == int(r.sum())
    assert (s[r == 0] == 0).all()
    assert (c.Bkw.sum(1) == c.Bk).all()


def test_association_generator_is_doubly_stochastic():
    G, V = 3, 50
    for S, eps in [(1, 0.0), (2, 0.2), (4, 0.3), (8, 0.5)]:
        ro, src, p = synth.associations(G, V, S, eps, 7)
        assert np.diff(ro).max() <= S and np.diff(ro).min() >= 1
        P = np.zeros((G, V, V))
        for q in range(G * V):
            g, w = divmod(q, V)
            assert src[ro[q]] == w  # the word itself comes first
            assert len(set(src[ro[q]:ro[q + 1]].tolist())) == ro[q + 1] - ro[q]
            P[g, w, src[ro[q]:ro[q + 1]]] += p[ro[q]:ro[q + 1]]
        np.testing.assert_allclose(P.sum(2), 1.0, rtol=1e-12)
        np.testing.assert_allclose(P.sum(1), 1.0, rtol=1e-12)


def test_repair_gives_the_most_probable_source():
    # one group, V = 3; row 0 lists sources (2, 0, 1) with p (0.2, 0.5, 0.3)
    words, off, grp = _corpus([(0, [0, 0, 1])])
    row_off = [0, 3, 4, 5]
    src = [2, 0, 1, 1, 2]
    p = [0.2, 0.5, 0.3, 1.0, 1.0]
    m = oracle.AssocModel(words, off, grp, 1, 1, 3, **HYP, row_off=row_off, src=src, p=p)
    assert m.head_source(0, 0) == 1 and m.head_source(0, 1) == 0
    z = np.zeros(3, np.int32)
    r = np.zeros(3, np.uint8)
    s = np.zeros(3, np.uint8)
    c = m.rebuild(z, r, s)
    assert m.repair(z, r, s, c) == 2
    assert r.tolist() == [1, 0, 1] and s.tolist() == [1, 0, 0]
    assert c.Bkw[0].tolist() == [1, 1, 0]  # sources 0 (word 0's head) and 1 (word 1's)
    # ties: the first of the tied slots
    m2 = oracle.AssocModel(words, off, grp, 1, 1, 3, **HYP, row_off=row_off, src=src,
                           p=[0.4, 0.4, 0.2, 1.0, 1.0])
    assert m2.head_source(0, 0) == 0
