"""Pins of the oracle's sampler mechanics and sweep invariants.

* Exact enumeration: on a corpus of a few tokens the posterior over every
  (z, r) state is proportional to exp(joint), and the joint itself is pinned
  to the Chinese-restaurant process by tests/test_oracle_joint.py.  The long-run
  state frequencies of the oracle's sequential collapsed-Gibbs chain (Algorithm
  SPDP-Full-Gibbs with stored table indicators) must match it; this exercises
  the Philox uniforms, the removal/addition, the outcome order and the
  inverse-CDF draw.  The snapshot-parallel chain is an approximation of the
  thesis's GPU scheme; its distance is reported, not asserted.
* Invariants of the counts after every snapshot sweep.
* Determinism: the snapshot sweep does not depend on the number of threads.
"""
import itertools
import math
import os
import subprocess
import sys

import numpy as np
import pytest

import oracle
import synth


def enumerate_posterior(m):
    K, N = m.K, m.N
    nb = (2 * K) ** N
    p = np.zeros(nb)
    for code in range(nb):
        z = np.empty(N, np.int32)
        r = np.empty(N, np.uint8)
        x = code
        for i in range(N):
            dgt = x % (2 * K)
            x //= 2 * K
            z[i], r[i] = dgt // 2, 1 - (dgt % 2)
        c = m.rebuild(z, r)
        ll = m.loglik(z, r, c)
        p[code] = -math.inf if ll == -math.inf else ll
    fin = np.isfinite(p)
    out = np.zeros(nb)
    out[fin] = np.exp(p[fin] - p[fin].max())
    return out / out.sum()


CHAIN_CASES = [
    # (docs as (group, words), K, V, hypers)
    ([(0, [0, 1, 0]), (1, [0, 0])], 2, 2, dict(alpha=0.5, a=0.5, b=2.0, gamma=0.5)),
    ([(0, [0, 1]), (0, [1, 1]), (1, [1])], 2, 3, dict(alpha=0.2, a=0.0, b=1.0, gamma=0.2)),
    ([(0, [2, 2, 2, 0])], 2, 3, dict(alpha=1.0, a=0.8, b=0.5, gamma=1.0)),
]


@pytest.mark.parametrize("case", range(len(CHAIN_CASES)))
def test_sequential_chain_matches_exact_posterior(case):
    docs, K, V, hyp = CHAIN_CASES[case]
    words = np.array([w for _, d in docs for w in d], np.int32)
    doc_off = np.cumsum([0] + [len(d) for _, d in docs]).astype(np.int64)
    doc_group = np.array([g for g, _ in docs], np.int32)
    m = oracle.Model(words, doc_off, doc_group, int(doc_group.max()) + 1, K, V, **hyp)
    post = enumerate_posterior(m)
    z, r, c = m.initial_state(11)
    n_sweeps = 1_500_000
    hist = m.chain_histogram(c, z, r, 0, 10_000, seed=123, mode="sequential")  # burn-in
    hist = m.chain_histogram(c, z, r, 10_000, n_sweeps, seed=123, mode="sequential")
    freq = hist / hist.sum()
    tv = 0.5 * np.abs(freq - post).sum()
    assert tv < 0.01, tv
    # every visited state is a valid one
    assert np.all(post[hist > 0] > 0)
    # per-state agreement for the well-populated states
    big = post > 0.01
    np.testing.assert_allclose(freq[big], post[big], rtol=0.06)

    zs, rs, cs = m.initial_state(11)
    hs = m.chain_histogram(cs, zs, rs, 0, 200_000, seed=99, mode="snapshot")
    tv_snap = 0.5 * np.abs(hs / hs.sum() - post).sum()
    print(f"case {case}: states {int((post > 0).sum())}, TV sequential {tv:.4f}, "
          f"TV snapshot {tv_snap:.4f} (approximation, reported only)")


def check_invariants(m, z, r, c):
    K, G = m.K, m.G
    assert c.n.sum() == m.N
    assert np.all(c.t >= 0) and np.all(c.t <= c.n)
    assert np.array_equal(c.t > 0, c.n > 0)
    assert np.array_equal(c.Ngk, c.n.sum(axis=2))
    assert np.array_equal(c.Tgk, c.t.sum(axis=2))
    assert np.array_equal(c.Bkw, c.t.sum(axis=0))
    assert np.array_equal(c.Bk, c.Bkw.sum(axis=1))
    assert np.all((z >= 0) & (z < K))
    assert int(r.sum()) == int(c.t.sum())
    fresh = m.rebuild(z, r)
    for f in ("n", "t", "Ngk", "Tgk", "Bkw", "Bk"):
        assert np.array_equal(getattr(fresh, f), getattr(c, f))


def test_snapshot_sweeps_keep_invariants():
    wl = synth.workload(0)
    cp = synth.generate(wl, 0)
    m = oracle.Model(cp.words, cp.doc_off, cp.doc_group, cp.n_groups, wl.K, wl.vocab,
                     wl.alpha, wl.a, wl.b, wl.gamma)
    z, r, c = m.initial_state(0)
    check_invariants(m, z, r, c)
    lls = [m.loglik(z, r, c)]
    total_repaired = 0
    for s in range(8):
        changed, repaired = m.sweep(c, z, r, s, seed=42, mode="snapshot")
        total_repaired += repaired
        check_invariants(m, z, r, c)
        assert 0 < changed <= m.N
        lls.append(m.loglik(z, r, c))
    assert lls[-1] > lls[0]  # the chain moves towards the posterior mode region
    assert all(math.isfinite(x) for x in lls)


def test_empty_documents_and_single_token_docs():
    docs = [(0, []), (0, [1]), (1, []), (1, [0, 0, 1]), (0, [])]
    words = np.array([w for _, d in docs for w in d], np.int32)
    doc_off = np.cumsum([0] + [len(d) for _, d in docs]).astype(np.int64)
    doc_group = np.array([g for g, _ in docs], np.int32)
    m = oracle.Model(words, doc_off, doc_group, 2, 3, 2, 0.1, 0.5, 10.0, 0.01)
    z, r, c = m.initial_state(3)
    for s in range(5):
        m.sweep(c, z, r, s, seed=1, mode="snapshot")
        check_invariants(m, z, r, c)


def test_snapshot_sweep_independent_of_thread_count():
    code = r"""
import sys, numpy as np
sys.path.insert(0, sys.argv[1])
import oracle, synth
wl = synth.workload(0)
cp = synth.generate(wl, 0)
m = oracle.Model(cp.words, cp.doc_off, cp.doc_group, cp.n_groups, wl.K, wl.vocab,
                 wl.alpha, wl.a, wl.b, wl.gamma)
z, r, c = m.initial_state(0)
for s in range(3):
    m.sweep(c, z, r, s, seed=7, mode="snapshot")
print(oracle.num_threads(), int(np.int64(z.astype(np.int64) * 2 + r).sum() % 1000003),
      hash(z.tobytes() + r.tobytes()))
"""
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    outs = []
    for th in ("1", "4"):
        env = dict(os.environ, OMP_NUM_THREADS=th, PYTHONHASHSEED="0")
        res = subprocess.run([sys.executable, "-c", code, root], env=env, capture_output=True,
                             text=True, check=True)
        outs.append(res.stdout.split())
    assert outs[0][0] == "1" and outs[1][0] == "4"
    assert outs[0][1:] == outs[1][1:]
