"""GPU parity of the model with word associations (non-identity
transformation matrices P^g) against the fp64 oracle, through the C ABI.

* Identity lists (one source per row, the word itself, p = 1) give the same
  chain as the plain library state.
* Initial state (z, r, source slot) and counts bit-exact; per-sweep parity
  with the protocol of tests/parity.py (counts bit-exact, conditionals within
  1e-5, samples identical on >= 99.99% of tokens with every first mismatch at a
  CDF boundary, update and repair bit-exact); source lists of 1..8 entries,
  K at the lane-layout boundaries, the 32-bit shadow-base path.
* Joint to 1e-6, estimates to fp64 rounding, held-out fold-in topics identical
  (1, 2, 4 and 8 source slots; 1 to 12 topics per lane).
* Checkpoint/resume with slots; invalid slots rejected.
Each test prints the case it runs before touching the GPU.
"""
import numpy as np
import pytest

import synth
from paper_1510_06549_amd import spdp as sp
from tests import parity

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)


class W:
    def __init__(self, K, alpha=0.1, a=0.5, b=10.0, gamma=0.01):
        self.K, self.alpha, self.a, self.b, self.gamma = K, alpha, a, b, gamma


def corpus_from_docs(docs, vocab):
    words = np.array([w for _, d in docs for w in d], np.int32)
    doc_off = np.cumsum([0] + [len(d) for _, d in docs]).astype(np.int64)
    doc_group = np.array([g for g, _ in docs], np.int32)
    return synth.Corpus(words, doc_off, doc_group, np.zeros_like(words),
                        np.zeros(len(words), np.uint8), int(doc_group.max()) + 1, vocab)


@pytest.fixture(scope="module")
def corpora():
    return {i: synth.generate(synth.workload(i), 0) for i in (0, 1, 2)}


def identity_lists(G, V):
    return (np.arange(G * V + 1, dtype=np.int64), np.tile(np.arange(V, dtype=np.int32), G),
            np.ones(G * V))


def test_identity_lists_give_the_plain_chain(corpora):
    wl = synth.workload(1)
    say(f"identity associations vs the plain state, workload {wl.name}")
    cp = corpora[1]
    plain, _ = parity.make_pair(cp, wl, init_seed=2)
    ident, _ = parity.make_pair(cp, wl, init_seed=2, assoc=identity_lists(cp.n_groups, cp.vocab))
    assert ident.S == 1 and plain.S == 0
    for sw in range(4):
        plain.sweep(sw, 31)
        ident.sweep(sw, 31)
        za, ra = plain.assignments()
        zb, rb = ident.assignments()
        agree = float(np.mean((za == zb) & (ra == rb)))
        say(f"  sweep {sw}: agreement {agree}")
        assert agree >= parity.MATCH_FRAC
        if agree == 1.0:
            for x, y in zip(plain.totals(), ident.totals()):
                assert np.array_equal(x, y)
    assert not ident.slots().any()
    lp, li = plain.loglik(), ident.loglik()
    assert abs(lp - li) <= 1e-12 * abs(lp)
    plain.close()
    ident.close()


ASSOC_CASES = [(0, 4, 0.3, 12), (1, 4, 0.3, 4), (2, 4, 0.3, 2), (0, 2, 0.5, 6), (0, 8, 0.4, 6),
               (1, 3, 0.2, 3)]


@pytest.mark.parametrize("idx", [0, 1, 2])
def test_initial_state_bit_exact(corpora, idx):
    wl = synth.workload(idx)
    say(f"initial state with associations, workload {wl.name}")
    cp = corpora[idx]
    assoc = synth.associations(cp.n_groups, cp.vocab, 4, 0.3, idx)
    s, m = parity.make_pair(cp, wl, init_seed=5, assoc=assoc)
    z0, r0, s0, c0 = m.initial_state(5)
    zg, rg = s.assignments()
    sg = s.slots()
    assert np.array_equal(zg, z0) and np.array_equal(rg, r0) and np.array_equal(sg, s0)
    parity.assert_counts_equal(s, c0)
    s.close()


@pytest.mark.parametrize("idx,S,eps,sweeps", ASSOC_CASES)
def test_sweeps_parity(corpora, idx, S, eps, sweeps):
    wl = synth.workload(idx)
    cp = corpora[idx]
    assoc = synth.associations(cp.n_groups, cp.vocab, S, eps, 10 + S)
    s, m = parity.make_pair(cp, wl, init_seed=1, assoc=assoc)
    assert s.S == m.S
    for sw in range(sweeps):
        say(f"association sweep parity, workload {wl.name}, S = {S}, sweep {sw}")
        rep, changed, repaired = parity.one_step(s, m, sw, seed=4048 + idx)
        say(f"  {rep} changed={changed} repaired={repaired}")
        assert changed > 0
    s.close()


@pytest.mark.parametrize("idx", [0, 1])
def test_loglik_parity(corpora, idx):
    wl = synth.workload(idx)
    say(f"association loglik parity, workload {wl.name}")
    cp = corpora[idx]
    assoc = synth.associations(cp.n_groups, cp.vocab, 4, 0.3, 3)
    s, m = parity.make_pair(cp, wl, init_seed=3, assoc=assoc)
    for sw in range(3):
        st = parity.state_of(s, m)
        ll_o = m.loglik(*st, m.rebuild(*st))
        ll_g = s.loglik()
        say(f"  sweep {sw}: gpu {ll_g!r} oracle {ll_o!r}")
        assert abs(ll_g - ll_o) <= 1e-6 * abs(ll_o)
        s.sweep(sw, 78)
    s.close()


def _ragged_assoc(G, V, rng, smax):
    """Source lists of random lengths 1..smax (the word itself first), random
    positive p, so rows of several lengths and padding slots meet."""
    row_off, src, p = [0], [], []
    for _ in range(G):
        for w in range(V):
            n = int(rng.integers(1, smax + 1))
            others = rng.choice(np.delete(np.arange(V), w), size=n - 1, replace=False)
            src += [w] + [int(v) for v in others]
            p += list(rng.uniform(0.05, 1.0, size=n))
            row_off.append(len(src))
    return (np.array(row_off, np.int64), np.array(src, np.int32), np.array(p, np.float64))


@pytest.mark.parametrize("K,smax", [(1, 3), (2, 8), (63, 5), (64, 1), (65, 2), (129, 4),
                                    (257, 7), (500, 4), (513, 3), (769, 2), (1024, 8)])
def test_topic_counts_and_list_lengths(K, smax):
    say(f"associations, K = {K}, lists of 1..{smax} sources")
    rng = np.random.default_rng(K + 100 * smax)
    docs = [(d % 2, list(rng.zipf(1.3, size=int(rng.integers(1, 120))) % 200)) for d in range(100)]
    cp = corpus_from_docs(docs, vocab=200)
    wl = W(K=K, alpha=0.2, a=0.6, b=5.0, gamma=0.05)
    assoc = _ragged_assoc(cp.n_groups, cp.vocab, rng, smax)
    s, m = parity.make_pair(cp, wl, assoc=assoc)
    for sw in range(3):
        rep, ch, rp = parity.one_step(s, m, sw, 5 + K)
    st = parity.state_of(s, m)
    ll_o = m.loglik(*st, m.rebuild(*st))
    assert abs(s.loglik() - ll_o) <= 1e-6 * abs(ll_o)
    s.close()


def test_shadow_base_counts_beyond_16_bits():
    """66 000 distinct words, each listing source 0 only, all seated as heads of
    topic 0: every head has source 0, so B[0][0] = 66 000 and the sampler reads
    the 32-bit shadow-base rows."""
    say("associations: shadow-base count beyond 16 bits")
    V = 66000
    words = np.arange(V, dtype=np.int32)
    doc_off = np.arange(0, V + 1, 1000, dtype=np.int64)
    doc_group = np.zeros(len(doc_off) - 1, np.int32)
    cp = synth.Corpus(words, doc_off, doc_group, np.zeros_like(words),
                      np.zeros(V, np.uint8), 1, V)
    assoc = (np.arange(V + 1, dtype=np.int64), np.zeros(V, np.int32), np.ones(V))
    wl = W(K=2, alpha=0.5, a=0.3, b=50.0, gamma=0.1)
    s, m = parity.make_pair(cp, wl, assoc=assoc)
    s.set_assignments(np.zeros(V, np.int32), np.ones(V, np.uint8), np.zeros(V, np.uint8))
    _, _, B, _ = s.totals()
    assert B[0, 0] == V and B.sum() == V
    rep, ch, rp = parity.one_step(s, m, 0, 21)
    say(f"  {rep}")
    s.close()


@pytest.mark.parametrize("idx", [0, 1])
def test_estimates_match_oracle(corpora, idx):
    wl = synth.workload(idx)
    say(f"association estimates, workload {wl.name}")
    cp = corpora[idx]
    assoc = synth.associations(cp.n_groups, cp.vocab, 4, 0.3, 9)
    s, m = parity.make_pair(cp, wl, init_seed=1, assoc=assoc)
    for sw in range(3):
        s.sweep(sw, 17)
    st = parity.state_of(s, m)
    c = m.rebuild(*st)
    th_o, p0_o, pg_o = m.estimates(st[0], c)
    th, p0, pg = s.estimates()
    np.testing.assert_allclose(th, th_o, rtol=1e-13)
    np.testing.assert_allclose(p0, p0_o.T, rtol=1e-13)
    np.testing.assert_allclose(pg, pg_o.transpose(0, 2, 1), rtol=1e-12)
    np.testing.assert_allclose(pg.sum(1), 1.0, rtol=1e-12)
    s.close()


@pytest.mark.parametrize("idx", [0, 1])
def test_heldout_matches_oracle(idx):
    wl = synth.workload(idx)
    say(f"association held-out fold-in, workload {wl.name}")
    cp = synth.generate(wl, 2)
    train, test = synth.split_heldout(cp, 0.1)
    assoc = synth.associations(cp.n_groups, cp.vocab, 4, 0.3, 4)
    s, m = parity.make_pair(train, wl, assoc=assoc)
    for sw in range(4):
        s.sweep(sw, 23)
    st = parity.state_of(s, m)
    c = m.rebuild(*st)
    _, _, pg_o = m.estimates(st[0], c)
    tot_o, zt_o, _ = m.heldout(pg_o, test.words, test.doc_off, test.doc_group, 10, 6)
    ppl, tot, zt = s.heldout(test.words, test.doc_off, test.doc_group, 10, 6)
    agree = float(np.mean(zt == zt_o)) if zt.size else 1.0
    say(f"  perplexity {ppl}, oracle total {tot_o}, library total {tot}, agreement {agree}")
    assert agree >= parity.MATCH_FRAC
    assert abs(tot - tot_o) <= 1e-9 * abs(tot_o)
    s.close()


@pytest.mark.parametrize("K,S", [(10, 1), (130, 2), (500, 4), (700, 4), (200, 8), (500, 8)])
def test_heldout_source_and_topic_layouts(K, S):
    """The fold-in's source-count and lane-layout instances (1, 2, 4 and 8
    source slots; 1 to 12 topics per lane), with and without the one-token
    prefetch (four sources past K = 512 and eight past K = 256 load each
    token's rows, then use them)."""
    w0 = synth.workload(0)
    say(f"association held-out fold-in, K = {K}, {S} sources per word")
    cp = synth.generate(w0, 3)
    train, test = synth.split_heldout(cp, 0.1)
    assoc = synth.associations(cp.n_groups, cp.vocab, S, 0.3 if S > 1 else 0.0, 8)
    s, m = parity.make_pair(train, W(K, w0.alpha, w0.a, w0.b, w0.gamma), assoc=assoc)
    for sw in range(3):
        s.sweep(sw, 29)
    st = parity.state_of(s, m)
    c = m.rebuild(*st)
    _, _, pg_o = m.estimates(st[0], c)
    tot_o, zt_o, _ = m.heldout(pg_o, test.words, test.doc_off, test.doc_group, 6, 11)
    ppl, tot, zt = s.heldout(test.words, test.doc_off, test.doc_group, 6, 11)
    agree = float(np.mean(zt == zt_o))
    say(f"  {test.n_tokens} test tokens, agreement {agree}, totals {tot} / {tot_o}")
    assert agree >= parity.MATCH_FRAC
    assert abs(tot - tot_o) <= 1e-9 * abs(tot_o)
    s.close()


def test_resume_with_slots_and_bad_slots_rejected(corpora):
    wl = synth.workload(0)
    say("association checkpoint/resume and invalid slots")
    cp = corpora[0]
    assoc = synth.associations(cp.n_groups, cp.vocab, 4, 0.3, 5)
    a, m = parity.make_pair(cp, wl, init_seed=9, assoc=assoc)
    for sw in range(3):
        a.sweep(sw, 55)
    z, r, sl = parity.state_of(a, m)
    c, _ = parity.make_pair(cp, wl, init_seed=123, assoc=assoc)
    c.set_assignments(z, r, sl)
    for sw in range(3, 6):
        a.sweep(sw, 55)
        c.sweep(sw, 55)
    for x, y in zip(parity.state_of(a, m), parity.state_of(c, m)):
        assert np.array_equal(x, y)
    # repair of an all-r = 0 state gives heads the most probable source
    rng = np.random.default_rng(0)
    z = rng.integers(0, wl.K, size=cp.n_tokens).astype(np.int32)
    r = np.zeros(cp.n_tokens, np.uint8)
    sl = np.zeros(cp.n_tokens, np.uint8)
    c.set_assignments(z, r, sl)
    zo, ro, so = z.copy(), r.copy(), sl.copy()
    co = m.rebuild(zo, ro, so)
    m.repair(zo, ro, so, co)
    for x, y in zip(parity.state_of(c, m), (zo, ro, so)):
        assert np.array_equal(x, y)
    parity.assert_counts_equal(c, co)
    # a head whose slot is just past its row's list
    lens = np.diff(assoc[0])
    q = cp.doc_group[np.searchsorted(cp.doc_off, np.arange(cp.n_tokens), "right") - 1] \
        * cp.vocab + cp.words
    short = np.flatnonzero(lens[q] < 4)
    i = int(short[0]) if short.size else 0
    z2, r2, s2 = parity.state_of(a, m)
    r2[i] = 1
    s2[i] = lens[q[i]]
    with pytest.raises(sp.SpdpError) as e:
        a.set_assignments(z2, r2, s2)
    assert e.value.code == sp.SPDP_E_ARG
    for x in (a, c):
        x.close()
