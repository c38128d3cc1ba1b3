"""The synthetic corpus generator: shape, validity and determinism."""
import math

import numpy as np

import synth


def test_shapes_and_ranges():
    for idx in (0, 1):
        wl = synth.workload(idx)
        cp = synth.generate(wl, 0)
        D = wl.n_groups * wl.docs_per_group
        assert cp.doc_off.shape == (D + 1,) and cp.doc_off[0] == 0
        assert np.all(np.diff(cp.doc_off) > 0)
        assert np.all((cp.words >= 0) & (cp.words < wl.vocab))
        assert np.all((cp.z_true >= 0) & (cp.z_true < wl.K))
        mean_len = cp.n_tokens / D
        assert abs(mean_len - wl.doc_len_mean) < 4 * math.sqrt(wl.doc_len_mean / D) + 0.5
        assert np.array_equal(np.unique(cp.doc_group), np.arange(wl.n_groups))


def test_deterministic():
    wl = synth.workload(0)
    a = synth.generate(wl, 3)
    b = synth.generate(wl, 3)
    c = synth.generate(wl, 4)
    assert np.array_equal(a.words, b.words) and np.array_equal(a.z_true, b.z_true)
    assert not np.array_equal(a.words, c.words)


def test_restaurant_table_counts_match_pyp_expectation():
    # Mean number of tables in a restaurant of n customers under PYP(a, b):
    # (b/a)[(b+a)_n/(b)_n - 1]; compare the generator's average over restaurants.
    wl = synth.workload(1)
    cp = synth.generate(wl, 0)
    g = np.repeat(cp.doc_group, np.diff(cp.doc_off))
    key = g.astype(np.int64) * wl.K + cp.z_true
    n = np.bincount(key, minlength=wl.n_groups * wl.K)
    t = np.bincount(key, weights=cp.r_true, minlength=wl.n_groups * wl.K)
    a, b = wl.a, wl.b
    exp_t = []
    for nn in n:
        if nn == 0:
            exp_t.append(0.0)
            continue
        lr = sum(math.log((b + a + j) / (b + j)) for j in range(nn))
        exp_t.append((b / a) * (math.exp(lr) - 1.0))
    exp_t = np.array(exp_t)
    mask = n > 0
    ratio = t[mask].sum() / exp_t[mask].sum()
    assert abs(ratio - 1.0) < 0.05, ratio


def test_true_shadow_base_is_the_law_of_new_tables():
    # Words served at new tables (r = 1) are draws from phi0 of their topic;
    # pooled over topics, the rank of such a word in its topic's law follows
    # the Zipf(s) pmf.  Chi-square over the first 30 ranks and a tail bucket.
    wl = synth.workload(1)
    cp = synth.generate(wl, 5)
    phi0 = synth.true_phi0(wl, 5)
    assert phi0.shape == (wl.K, wl.vocab)
    np.testing.assert_allclose(phi0.sum(1), 1.0, rtol=1e-12)
    rank = np.empty_like(phi0, dtype=np.int64)
    for k in range(wl.K):
        rank[k, np.argsort(-phi0[k], kind="stable")] = np.arange(wl.vocab)
    sel = cp.r_true == 1
    rk = rank[cp.z_true[sel], cp.words[sel]]
    zipf = np.arange(1, wl.vocab + 1, dtype=np.float64) ** -wl.zipf_s
    zipf /= zipf.sum()
    n = rk.size
    obs = np.append(np.bincount(rk, minlength=wl.vocab)[:30], (rk >= 30).sum())
    exp = np.append(zipf[:30], zipf[30:].sum()) * n
    chi2 = float(((obs - exp) ** 2 / exp).sum())
    assert chi2 < 70.0, chi2  # 30 dof: p ~ 1e-4
    # the law is the generator's for this seed only
    assert not np.array_equal(np.argmax(phi0, 1), np.argmax(synth.true_phi0(wl, 6), 1))
