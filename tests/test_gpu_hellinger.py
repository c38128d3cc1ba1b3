"""GPU Hellinger distances between topic models and the topic alignment,
against the oracle.

* spdp_hellinger equals the oracle's distances (|H^2 difference| <= 1e-12) on
  random laws with topic counts and outcome counts that span several 64-wide
  tiles and leave ragged tails, on host and on device buffers, with the
  state's own phi0 as the first model, and at the largest workload's shape
  (K = 500 topics over V = 100 000 words) on sampled rows.
* spdp_align_topics reaches the oracle's least total distance with a valid
  one-to-one matching (square and rectangular), recovers a planted
  permutation, and rejects bad arguments.
"""
import itertools

import numpy as np
import pytest
import torch

import oracle
import synth
from paper_1510_06549_amd import spdp as sp
from tests import parity

pytestmark = pytest.mark.gpu

TOL_H2 = 1e-12


def say(*a):
    print(*a, flush=True)


def _laws(rng, k, V, conc):
    """k random distributions over V outcomes, as columns of a [V, k] array."""
    return np.ascontiguousarray(rng.dirichlet(np.full(V, conc), size=k).T)


@pytest.fixture(scope="module")
def state():
    cp = synth.generate(synth.workload(0), 0)
    wl = synth.workload(0)
    s = sp.Sampler(cp.words, cp.doc_off, cp.doc_group, cp.n_groups, cp.vocab, wl.K, wl.alpha,
                   wl.a, wl.b, wl.gamma)
    yield s
    s.close()


@pytest.mark.parametrize("kp,kq,V", [(10, 10, 1000), (65, 129, 3001), (1, 200, 17),
                                     (200, 63, 20000), (64, 64, 16), (3, 2, 1)])
def test_hellinger_matches_oracle(state, kp, kq, V):
    say(f"hellinger kp={kp} kq={kq} V={V}")
    rng = np.random.default_rng(kp * 7 + kq * 3 + V)
    P = _laws(rng, kp, V, 0.05)
    Q = _laws(rng, kq, V, 0.05)
    Q[:, 0] = P[:, 0]  # an identical pair: distance 0
    H = state.hellinger(Q, P)
    Ho = oracle.hellinger(P.T, Q.T)
    assert H.shape == (kp, kq)
    assert np.all(np.abs(H * H - Ho * Ho) <= TOL_H2), np.abs(H * H - Ho * Ho).max()
    assert np.all((H >= 0) & (H <= 1))
    # device buffers
    dev = torch.device("cuda:0")
    Pd, Qd = torch.from_numpy(P).to(dev), torch.from_numpy(Q).to(dev)
    Hd = torch.empty((kp, kq), dtype=torch.float64, device=dev)
    sp.spdp_hellinger(state.h, Pd, Qd, Hd)
    np.testing.assert_array_equal(Hd.cpu().numpy(), H)


def test_hellinger_of_the_state_phi0(state):
    say("hellinger of the state's phi0 against the generating law")
    wl = synth.workload(0)
    truth = synth.true_phi0(wl, 0)  # [K, V]
    H = state.hellinger(np.ascontiguousarray(truth.T))
    _, phi0, _ = state.estimates()
    Ho = oracle.hellinger(phi0.T, truth)
    assert np.all(np.abs(H * H - Ho * Ho) <= TOL_H2)


def test_hellinger_empty_shapes(state):
    say("hellinger empty shapes")
    rng = np.random.default_rng(0)
    Q = _laws(rng, 4, 9, 1.0)
    assert state.hellinger(Q, np.zeros((9, 0))).shape == (0, 4)
    assert state.hellinger(np.zeros((9, 0)), Q[:, :3]).shape == (3, 0)
    # no outcomes at all: nothing in common, distance 1
    H = state.hellinger(np.zeros((0, 2)), np.zeros((0, 3)))
    np.testing.assert_array_equal(H, np.ones((3, 2)))


def test_hellinger_rejects_bad_arguments(state):
    say("hellinger argument checks")
    q = np.full((5, 2), 0.2)
    out = np.empty((3, 2))
    with pytest.raises(sp.SpdpError):  # p = NULL needs kp = K and V of the state
        sp.spdp_hellinger(state.h, None, q, out)
    with pytest.raises(sp.SpdpError):
        sp.spdp_hellinger(state.h, np.full((5, sp.SPDP_MAX_K + 1), 0.2), q,
                          np.empty((sp.SPDP_MAX_K + 1, 2)))


def test_hellinger_at_the_largest_shape_sampled(state):
    # K = 500 topics over 100 000 words: the GPU computes all 250 000 pairs,
    # the oracle 12 sampled rows of them
    say("hellinger 500 x 500 over 100000 outcomes, sampled rows")
    rng = np.random.default_rng(99)
    V, K = 100_000, 500
    P = _laws(rng, K, V, 0.01)
    Q = _laws(rng, K, V, 0.01)
    Q[:, 7] = P[:, 7]
    H = state.hellinger(Q, P)
    rows = np.concatenate([[0, 7, 63, 64, 255, 499], rng.choice(K, 6, replace=False)])
    Ho = oracle.hellinger(P[:, rows].T, Q.T)
    assert np.all(np.abs(H[rows] ** 2 - Ho ** 2) <= TOL_H2)
    assert H[7, 7] < 1e-6


@pytest.mark.parametrize("kp,kq", [(5, 5), (6, 6), (3, 7), (1, 1), (40, 40), (200, 260), (500, 500)])
def test_align_topics_matches_oracle(kp, kq):
    say(f"align kp={kp} kq={kq}")
    rng = np.random.default_rng(kp * 1000 + kq)
    H = rng.random((kp, kq))
    match, total = sp.spdp_align_topics(H)
    mo, to = oracle.align_topics(H)
    assert len(set(match.tolist())) == kp and match.min() >= 0 and match.max() < kq
    assert abs(H[np.arange(kp), match].sum() - total) <= 1e-12 * max(1.0, total)
    assert abs(total - to) <= 1e-10 * max(1.0, to)
    if kq <= 7:
        best = min(sum(H[i, c[i]] for i in range(kp))
                   for c in itertools.permutations(range(kq), kp))
        assert abs(total - best) <= 1e-12


def test_align_topics_recovers_a_planted_permutation():
    rng = np.random.default_rng(3)
    P = rng.dirichlet(np.full(300, 0.1), size=50)
    perm = rng.permutation(50)
    H = oracle.hellinger(P, P[perm])
    match, total = sp.spdp_align_topics(H)
    assert total == 0.0
    np.testing.assert_array_equal(perm[match], np.arange(50))


def test_align_topics_rejects_bad_arguments():
    with pytest.raises(sp.SpdpError):
        sp.spdp_align_topics(np.zeros((3, 2)))
    bad = np.zeros((2, 2))
    bad[1, 0] = np.nan
    with pytest.raises(sp.SpdpError):
        sp.spdp_align_topics(bad)
    m, t = sp.spdp_align_topics(np.zeros((0, 4)))
    assert m.size == 0 and t == 0.0
