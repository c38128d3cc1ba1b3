"""Pins of the oracle's joint and conditionals against the generative process.

* The oracle's joint log p(W, Z, R) (the collapsed joint of the thesis's
  blocked-Gibbs derivation, P = I), summed over every table-indicator labelling
  R, must equal p(W, Z) computed by brute force from the Chinese-restaurant
  definition of the process (tests/brute.py) -- a different route through the
  mathematics, which pins the Stirling, binomial, PYP-normaliser, shadow-base
  and document terms together.
* The oracle's per-token weights (Eq. SPDP-sampling-w-z-r0 / -r1) must equal
  ratios of that joint (the predictive = ratio of joints identity of the
  thesis's collapsed-Gibbs background), including exact zeros.
"""
import itertools
import math

import numpy as np
import pytest

import oracle
from tests import brute


def tiny_corpus():
    # G = 2 groups, V = 3 words, 4 documents, 10 tokens; word 0 appears four
    # times in group 0, so cells reach n = 3 after a removal
    docs = [(0, [0, 1, 0]), (0, [0, 1, 0]), (1, [2, 0]), (1, [0, 2])]
    words = np.array([w for _, d in docs for w in d], dtype=np.int32)
    doc_off = np.cumsum([0] + [len(d) for _, d in docs]).astype(np.int64)
    doc_group = np.array([g for g, _ in docs], dtype=np.int32)
    return words, doc_off, doc_group


def wider_corpus():
    # 18 tokens, word 0 six times in group 0: cells up to n = 5 after removal
    docs = [(0, [0, 1, 0, 0]), (0, [0, 1, 2, 0]), (0, [0]), (1, [2, 0, 2]), (1, [0, 2, 2, 1]),
            (1, [2])]
    words = np.array([w for _, d in docs for w in d], dtype=np.int32)
    doc_off = np.cumsum([0] + [len(d) for _, d in docs]).astype(np.int64)
    doc_group = np.array([g for g, _ in docs], dtype=np.int32)
    return words, doc_off, doc_group


HYPERS = [
    dict(alpha=0.1, a=0.5, b=10.0, gamma=0.01),
    dict(alpha=0.7, a=0.0, b=1.5, gamma=0.3),
    dict(alpha=0.05, a=0.8, b=0.7, gamma=1.2),
]


def make_model(K, hyp, corpus=None):
    words, doc_off, doc_group = corpus if corpus is not None else tiny_corpus()
    return oracle.Model(words, doc_off, doc_group, n_groups=int(doc_group.max()) + 1, K=K,
                        vocab=3, **hyp)


def loglik_of(m, z, r):
    c = m.rebuild(z, r)
    return m.loglik(z, r, c)


@pytest.mark.parametrize("hyp", HYPERS)
def test_joint_summed_over_labellings_equals_crp_marginal(hyp):
    K = 2
    m = make_model(K, hyp)
    rng = np.random.default_rng(1)
    for _ in range(4):
        z = rng.integers(0, K, size=m.N).astype(np.int32)
        acc = []
        for bits in itertools.product([0, 1], repeat=m.N):
            r = np.array(bits, dtype=np.uint8)
            ll = loglik_of(m, z, r)
            if ll != -math.inf:
                acc.append(ll)
        acc = np.array(acc)
        mx = acc.max()
        log_sum = mx + math.log(np.exp(acc - mx).sum())
        want = brute.log_p_WZ(list(m.words), list(m.doc_off), list(m.doc_group), list(z), m.G,
                              K, m.V, hyp["alpha"], hyp["a"], hyp["b"], hyp["gamma"])
        assert log_sum == pytest.approx(want, rel=1e-12, abs=1e-12)


def random_valid_state(m, rng):
    z = rng.integers(0, m.K, size=m.N).astype(np.int32)
    r = rng.integers(0, 2, size=m.N).astype(np.uint8)
    c = m.rebuild(z, r)
    m.repair(z, r, c)
    return z, r, c


@pytest.mark.parametrize("hyp", HYPERS)
@pytest.mark.parametrize("K", [1, 2, 3])
def test_conditionals_are_joint_ratios(hyp, K):
    m = make_model(K, hyp, corpus=wider_corpus())
    rng = np.random.default_rng(7 + K)
    checked = 0
    for _ in range(12):
        z, r, c = random_valid_state(m, rng)
        base_ll = m.loglik(z, r, c)
        assert math.isfinite(base_ll)
        for d in range(m.D):
            g = int(m.doc_group[d])
            crow = np.bincount(z[m.doc_off[d]:m.doc_off[d + 1]], minlength=K)
            for i in range(m.doc_off[d], m.doc_off[d + 1]):
                w = m.token_weights(c, crow, g, m.words[i], z[i], r[i])
                lls = np.empty(2 * K)
                for j in range(2 * K):
                    z2, r2 = z.copy(), r.copy()
                    z2[i], r2[i] = j // 2, 1 - (j % 2)
                    lls[j] = loglik_of(m, z2, r2)
                if w is None:
                    # sole head of a cell with other customers: every other
                    # outcome is impossible, the current one is certain
                    cur = 2 * z[i] + (1 - r[i])
                    assert all(lls[j] == -math.inf for j in range(2 * K) if j != cur)
                    assert math.isfinite(lls[cur])
                    continue
                fin = np.isfinite(lls)
                assert np.array_equal(w > 0, fin), (w, lls)
                p_joint = np.zeros(2 * K)
                p_joint[fin] = np.exp(lls[fin] - lls[fin].max())
                p_joint /= p_joint.sum()
                np.testing.assert_allclose(w / w.sum(), p_joint, rtol=1e-10, atol=1e-14)
                checked += 1
    assert checked > 50


def test_sole_head_rule_fires():
    # token 0 and 2 share (g=0, k=0, w=0); token 0 is the only head.
    K = 2
    m = make_model(K, HYPERS[0])
    z = np.zeros(m.N, dtype=np.int32)
    r = np.zeros(m.N, dtype=np.uint8)
    c = m.rebuild(z, r)
    m.repair(z, r, c)
    assert r[0] == 1 and r[2] == 0  # smallest index promoted
    crow = np.bincount(z[0:3], minlength=K)
    assert m.token_weights(c, crow, 0, 0, 0, 1) is None
    # the non-head may move
    assert m.token_weights(c, crow, 0, 0, 0, 0) is not None


@pytest.mark.parametrize("hyp", HYPERS)
def test_single_token_closed_form(hyp):
    # One token: after removal everything is empty, so W0 = 0 and
    # W1(k) = alpha * (b/b) * gamma/(V gamma) * 1 = alpha / V for every k.
    K, V = 4, 7
    m = oracle.Model(np.array([3], np.int32), np.array([0, 1], np.int64),
                     np.array([0], np.int32), n_groups=1, K=K, vocab=V, **hyp)
    z, r, c = m.initial_state(5)
    assert r[0] == 1
    w = m.token_weights(c, np.bincount(z, minlength=K), 0, 3, z[0], r[0])
    np.testing.assert_allclose(w[0::2], hyp["alpha"] / V, rtol=1e-15)
    assert np.all(w[1::2] == 0.0)


def test_loglik_generator_truth_beats_random_init():
    import synth

    wl = synth.workload(0)
    cp = synth.generate(wl, 0)
    m = oracle.Model(cp.words, cp.doc_off, cp.doc_group, cp.n_groups, wl.K, wl.vocab,
                     wl.alpha, wl.a, wl.b, wl.gamma)
    z0, r0, c0 = m.initial_state(0)
    zt, rt = cp.z_true.copy(), cp.r_true.copy()
    ct = m.rebuild(zt, rt)
    assert m.repair(zt, rt, ct) == 0  # the generator's state is valid
    assert m.loglik(zt, rt, ct) > m.loglik(z0, r0, c0)
