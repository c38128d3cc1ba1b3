"""Parity at the largest workload (250M tokens, K = 500), in the launch
configuration the benchmark times.

The oracle cannot run a whole sweep of this size in test time, so:
  * counts: the library's totals, shadow base and the count rows of two whole
    groups equal the oracle's rebuild of the library's state, bit for bit;
  * sampling: for documents sampled at the start, middle and end of the corpus
    the library's weights, uniforms and draws are compared with the oracle's
    one by one (same protocol as the small workloads), and the draws of 30 000
    whole documents (7.5 M tokens) with the oracle's sampling step;
  * update and repair: the library's state after the sweep equals the
    oracle's rebuild and repair of the library's sampled (pre-repair) state,
    for every token.
"""
import numpy as np
import pytest

import oracle
import synth
from tests import parity

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)


@pytest.mark.parametrize("warm", [1, 25])
def test_largest_workload_sampled_parity(warm):
    """warm = 1: the sweep after one warm-up sweep; warm = 25: the sweep after
    the benchmark's 5 warm-up and 20 timed sweeps (same seed and sweep
    numbers), the state the benchmark measures; there the joint is checked
    too (Eq. SPDP-Blocked-Gibbs-Joint-Prob, P = I)."""
    import torch

    wl = synth.workload("g20-d50000-k500")
    say(f"full-size parity, workload {wl.name}, after {warm} sweep(s): generating corpus")
    cp = synth.generate(wl, 0)
    s = parity.sp.Sampler(cp.words, cp.doc_off, cp.doc_group, cp.n_groups, wl.vocab, wl.K,
                          wl.alpha, wl.a, wl.b, wl.gamma, init_seed=0,
                          hip_stream=torch.cuda.current_stream().cuda_stream)
    seed = 1000
    say(f"  {warm} warm-up sweep(s)")
    for sw in range(warm):
        s.sweep(sw, seed)
    z, r = s.assignments()
    say("  oracle model and dense rebuild")
    m = oracle.Model(cp.words, cp.doc_off, cp.doc_group, cp.n_groups, wl.K, wl.vocab, wl.alpha,
                     wl.a, wl.b, wl.gamma)
    c = m.rebuild(z, r)
    assert m.repair(z.copy(), r.copy(), c.copy()) == 0, "library state has a cell without a head"

    # counts of the library's state
    say("  counts")
    N, T, B, Bk = s.totals()
    assert np.array_equal(N, c.Ngk) and np.array_equal(T, c.Tgk)
    assert np.array_equal(B, c.Bkw.T) and np.array_equal(Bk, c.Bk)
    for g in (0, cp.n_groups - 1):
        n_g, t_g = s.counts(g, g + 1)
        assert np.array_equal(n_g[0], c.n[g]), f"n of group {g}"
        assert np.array_equal(t_g[0], c.t[g]), f"t of group {g}"
    del n_g, t_g
    if warm > 1:
        say("  joint of the library's state against the oracle's")
        ll_g = s.loglik()
        ll_o = m.loglik(z, r, c)
        say(f"    library {ll_g!r} oracle {ll_o!r} rel {abs(ll_g - ll_o) / abs(ll_o):.3e}")
        assert abs(ll_g - ll_o) <= parity.LL_RTOL * abs(ll_o)

    # sampled documents, one by one against the oracle
    sweep = warm
    zo, ro = z.copy(), r.copy()
    for d0 in (0, m.D // 2 + 7, m.D - 150):
        d1 = d0 + 150
        tb, te = int(m.doc_off[d0]), int(m.doc_off[d1])
        say(f"  documents [{d0}, {d1}): tokens [{tb}, {te})")
        w_g, u_g, zr_g = s.conditionals(sweep, seed, tb, te)
        _, w_o, u_o, skip_o = m.sample_docs(c, zo, ro, sweep, seed, d0, d1, trace=(tb, te))
        skip_o = skip_o.astype(bool)
        zg, rg = zr_g >> 1, (zr_g & 1).astype(np.uint8)
        same = (zg == zo[tb:te]) & (rg == ro[tb:te])
        assert same.mean() >= parity.MATCH_FRAC, same.mean()
        assert np.array_equal(u_g < 0, skip_o)
        sel = same & ~skip_o  # identical draws, so identical document rows up to here
        ok = np.ones(te - tb, dtype=bool)
        # tokens after a document's first mismatch are excluded from weight checks
        doc = np.repeat(np.arange(d1 - d0), np.diff(m.doc_off[d0:d1 + 1]))
        for i in np.flatnonzero(~same):
            ok &= ~((doc == doc[i]) & (np.arange(te - tb) > i))
        sel &= ok
        wo, wg = w_o[sel], w_g[sel].astype(np.float64)
        nz = wo != 0
        assert np.all(wg[~nz] == 0)
        assert np.max(np.abs(wg[nz] - wo[nz]) / wo[nz]) <= parity.W_RTOL
        assert np.array_equal(u_g[sel].astype(np.float64), u_o[sel])
        del w_g, w_o

    # the draws of 30 000 whole documents (7.5 M tokens) against the oracle's
    # sampling step, without traces
    zr_pre = s.sampled(sweep, seed)
    zgp, rgp = (zr_pre >> 1).astype(np.int32), (zr_pre & 1).astype(np.uint8)
    zo, ro = z.copy(), r.copy()
    for d0 in (0, m.D // 2 - 5000, m.D - 10000):
        d1 = d0 + 10000
        tb, te = int(m.doc_off[d0]), int(m.doc_off[d1])
        say(f"  draws of documents [{d0}, {d1}) (tokens [{tb}, {te})) against the oracle")
        m.sample_docs(c, zo, ro, sweep, seed, d0, d1)
        same = (zgp[tb:te] == zo[tb:te]) & (rgp[tb:te] == ro[tb:te])
        say(f"    {int((~same).sum())} of {te - tb} differ")
        assert same.mean() >= parity.MATCH_FRAC, same.mean()
    del zgp, rgp, zo, ro

    # the whole sweep: library state after update and repair vs the oracle's
    # rebuild and repair of the library's sampled state
    say("  whole sweep: update and repair of all tokens")
    s.sweep(sweep, seed)
    zs, rs = s.assignments()
    zp, rp = (zr_pre >> 1).astype(np.int32), (zr_pre & 1).astype(np.uint8)
    c2 = m.rebuild(zp, rp, c)
    promoted = m.repair(zp, rp, c2)
    changed, repaired = s.stats()
    say(f"  promoted {promoted} (library {repaired}), changed {changed}")
    assert repaired == promoted
    assert np.array_equal(zs, zp) and np.array_equal(rs, rp)
    N, T, B, Bk = s.totals()
    assert np.array_equal(N, c2.Ngk) and np.array_equal(T, c2.Tgk)
    assert np.array_equal(B, c2.Bkw.T) and np.array_equal(Bk, c2.Bk)
    s.close()
