"""Pins of the oracle's ordered sequential sweep, the exact counterpart of
the thesis's asynchronous GPU scheme (word order rearrangement; live counts
updated after every token).

* The interleaved visiting order follows the thesis's construction: round
  robin over the position inside the document, every document that is long
  enough contributing its token at each position (hand example, and a
  permutation that keeps each document's tokens in order on a generated
  corpus).
* With the identity order the ordered sweep is the sequential sweep exactly.
* With the interleaved order (and with a random order) the chain's long-run
  state frequencies match the exact posterior enumerated over every (z, r):
  single-site Gibbs in any fixed scan order leaves the posterior invariant.
* The ordered sweep keeps every state valid: the repair has nothing to do.
"""
import numpy as np
import pytest

import oracle
import synth
from tests.test_oracle_chain import CHAIN_CASES, enumerate_posterior


def _model(docs, K, V, hyp):
    words = np.array([w for _, d in docs for w in d], np.int32)
    doc_off = np.cumsum([0] + [len(d) for _, d in docs]).astype(np.int64)
    doc_group = np.array([g for g, _ in docs], np.int32)
    return oracle.Model(words, doc_off, doc_group, int(doc_group.max()) + 1, K, V, **hyp)


def test_interleaved_order_hand_example():
    # document lengths 3, 0, 1, 2: positions 0 (docs 0, 2, 3), 1 (docs 0, 3), 2 (doc 0)
    m = _model([(0, [0, 1, 0]), (0, []), (1, [1]), (1, [0, 0])], 2, 2,
               dict(alpha=0.5, a=0.5, b=1.0, gamma=0.5))
    assert m.interleaved_order().tolist() == [0, 3, 4, 1, 5, 2]


def test_interleaved_order_on_a_corpus():
    cp = synth.generate(synth.workload(0), 2)
    wl = synth.workload(0)
    m = oracle.Model(cp.words, cp.doc_off, cp.doc_group, cp.n_groups, wl.K, cp.vocab, wl.alpha,
                     wl.a, wl.b, wl.gamma)
    order = m.interleaved_order()
    assert np.array_equal(np.sort(order), np.arange(cp.n_tokens))
    doc = np.searchsorted(cp.doc_off, order, "right") - 1
    pos = order - cp.doc_off[doc]
    # positions never decrease; within one position documents increase
    assert np.all(np.diff(pos) >= 0)
    same = np.diff(pos) == 0
    assert np.all(np.diff(doc)[same] > 0)


def test_identity_order_is_the_sequential_sweep():
    cp = synth.generate(synth.workload(0), 4)
    wl = synth.workload(0)
    m = oracle.Model(cp.words, cp.doc_off, cp.doc_group, cp.n_groups, wl.K, cp.vocab, wl.alpha,
                     wl.a, wl.b, wl.gamma)
    z1, r1, c1 = m.initial_state(3)
    z2, r2, c2 = m.initial_state(3)
    ident = np.arange(m.N, dtype=np.int32)
    for sw in range(3):
        a = m.sweep(c1, z1, r1, sw, 17, mode="sequential")
        b = m.sweep(c2, z2, r2, sw, 17, mode="ordered", order=ident)
        assert a[0] == b[0]
    assert np.array_equal(z1, z2) and np.array_equal(r1, r2)
    assert np.array_equal(c1.n, c2.n) and np.array_equal(c1.t, c2.t)


@pytest.mark.parametrize("case", range(len(CHAIN_CASES)))
@pytest.mark.parametrize("which", ["interleaved", "random"])
def test_ordered_chain_matches_exact_posterior(case, which):
    docs, K, V, hyp = CHAIN_CASES[case]
    m = _model(docs, K, V, hyp)
    post = enumerate_posterior(m)
    order = (m.interleaved_order() if which == "interleaved"
             else np.random.default_rng(case).permutation(m.N).astype(np.int32))
    z, r, c = m.initial_state(7)
    m.chain_histogram(c, z, r, 0, 10_000, seed=321, mode="ordered", order=order)
    hist = m.chain_histogram(c, z, r, 10_000, 1_500_000, seed=321, mode="ordered", order=order)
    freq = hist / hist.sum()
    tv = 0.5 * np.abs(freq - post).sum()
    assert tv < 0.01, tv
    assert np.all(post[hist > 0] > 0)
    big = post > 0.01
    np.testing.assert_allclose(freq[big], post[big], rtol=0.06)


def test_ordered_sweep_keeps_the_state_valid():
    cp = synth.generate(synth.workload(1), 1)
    wl = synth.workload(1)
    m = oracle.Model(cp.words, cp.doc_off, cp.doc_group, cp.n_groups, wl.K, cp.vocab, wl.alpha,
                     wl.a, wl.b, wl.gamma)
    z, r, c = m.initial_state(2)
    order = m.interleaved_order()
    for sw in range(2):
        m.sweep(c, z, r, sw, 5, mode="ordered", order=order)
    c2 = m.rebuild(z, r)
    for f in ("n", "t", "Ngk", "Tgk", "Bkw", "Bk"):
        assert np.array_equal(getattr(c, f), getattr(c2, f)), f
    assert m.repair(z, r, c2) == 0
    assert np.isfinite(m.loglik(z, r, c2))


def test_stale_totals_sweep_keeps_the_state_valid_and_differs_from_live():
    """The variant with the sums N_gk, T_gk, B_k held at their sweep-start
    values is not exact Gibbs (parity unpinned against the paper, which
    describes the drifting sums only in words); its sweep keeps the state
    valid, its live counts equal the rebuild, and it moves away from the live
    sweep once the sums have changed."""
    cp = synth.generate(synth.workload(0), 5)
    wl = synth.workload(0)
    m = oracle.Model(cp.words, cp.doc_off, cp.doc_group, cp.n_groups, wl.K, cp.vocab, wl.alpha,
                     wl.a, wl.b, wl.gamma)
    order = m.interleaved_order()
    z1, r1, c1 = m.initial_state(8)
    z2, r2, c2 = m.initial_state(8)
    for sw in range(2):
        m.sweep(c1, z1, r1, sw, 3, mode="ordered", order=order, stale_totals=True)
        m.sweep(c2, z2, r2, sw, 3, mode="ordered", order=order)
    c1r = m.rebuild(z1, r1)
    for f in ("n", "t", "Ngk", "Tgk", "Bkw", "Bk"):
        assert np.array_equal(getattr(c1, f), getattr(c1r, f)), f
    assert m.repair(z1, r1, c1r) == 0
    assert np.isfinite(m.loglik(z1, r1, c1r))
    assert not (np.array_equal(z1, z2) and np.array_equal(r1, r2))
