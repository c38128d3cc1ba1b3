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
