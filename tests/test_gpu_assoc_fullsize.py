"""Parity of the model with word associations at the largest workload (250M
tokens, K = 500, four sources per word, as `bench.py --assoc 4` runs it):
  * counts: totals, the source-keyed shadow base and the count rows of two
    whole groups equal the oracle's rebuild of the library's state;
  * sampling: weights, uniforms and draws of 40 documents at the start, middle
    and end of the corpus one by one, and the draws (topic, table indicator
    and source slot) of 6 000 whole documents against the oracle's sampling
    step;
  * update and repair: the library's state after the sweep equals the
    oracle's rebuild and repair of the library's sampled state, for every
    token, and so do the totals.
Each step prints what it runs before touching the GPU.
"""
import numpy as np
import pytest

import oracle
import synth
from tests import parity

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)


def test_largest_workload_with_associations():
    import torch

    wl = synth.workload("g20-d50000-k500")
    say(f"full-size parity with associations, workload {wl.name}: generating corpus")
    cp = synth.generate(wl, 0)
    assoc = synth.associations(cp.n_groups, cp.vocab, 4, 0.3, 0)
    s = parity.sp.Sampler(cp.words, cp.doc_off, cp.doc_group, cp.n_groups, wl.vocab, wl.K,
                          wl.alpha, wl.a, wl.b, wl.gamma, init_seed=0,
                          hip_stream=torch.cuda.current_stream().cuda_stream, assoc=assoc)
    seed = 2000
    say("  warm-up sweep")
    s.sweep(0, seed)
    z, r = s.assignments()
    sl = s.slots()
    say("  oracle model and dense rebuild")
    m = oracle.AssocModel(cp.words, cp.doc_off, cp.doc_group, cp.n_groups, wl.K, wl.vocab,
                          wl.alpha, wl.a, wl.b, wl.gamma, *assoc)
    c = m.rebuild(z, r, sl)

    say("  counts")
    N, T, B, Bk = s.totals()
    assert np.array_equal(N, c.Ngk) and np.array_equal(T, c.Tgk)
    assert np.array_equal(B, c.Bkw.T) and np.array_equal(Bk, c.Bk)
    for g in (0, cp.n_groups - 1):
        n_g, t_g = s.counts(g, g + 1)
        assert np.array_equal(n_g[0], c.n[g]), f"n of group {g}"
        assert np.array_equal(t_g[0], c.t[g]), f"t of group {g}"
    del n_g, t_g

    sweep = 1
    zr_pre = s.sampled(sweep, seed)
    zg, rg, sg = parity.unpack(zr_pre)
    zg = zg.astype(np.int32)
    for d0 in (0, m.D // 2 + 3, m.D - 40):
        d1 = d0 + 40
        tb, te = int(m.doc_off[d0]), int(m.doc_off[d1])
        say(f"  documents [{d0}, {d1}): weights, uniforms and draws of tokens [{tb}, {te})")
        w_g, u_g, zr_g = s.conditionals(sweep, seed, tb, te)
        assert np.array_equal(zr_g, zr_pre[tb:te])
        zt, rt, st = z.copy(), r.copy(), sl.copy()
        _, w_o, u_o, _ = m.sample_docs(c, zt, rt, st, sweep, seed, d0, d1, trace=(tb, te))
        same = (zg[tb:te] == zt[tb:te]) & (rg[tb:te] == rt[tb:te]) & (sg[tb:te] == st[tb:te])
        assert same.mean() >= parity.MATCH_FRAC, same.mean()
        doc = np.repeat(np.arange(d1 - d0), np.diff(m.doc_off[d0:d1 + 1]))
        ok = np.ones(te - tb, dtype=bool)
        for i in np.flatnonzero(~same):
            ok &= ~((doc == doc[i]) & (np.arange(te - tb) > i))
        wo, wgt = w_o[ok], w_g[ok].astype(np.float64)
        nz = wo != 0
        assert np.all(wgt[~nz] == 0)
        assert np.max(np.abs(wgt[nz] - wo[nz]) / wo[nz]) <= parity.W_RTOL
        assert np.array_equal(u_g[ok].astype(np.float64), u_o[ok])
        del w_g, w_o

    zo, ro, so = z.copy(), r.copy(), sl.copy()
    for d0 in (0, m.D // 2 - 1000, m.D - 2000):
        d1 = d0 + 2000
        tb, te = int(m.doc_off[d0]), int(m.doc_off[d1])
        say(f"  draws of documents [{d0}, {d1}) (tokens [{tb}, {te})) against the oracle")
        m.sample_docs(c, zo, ro, so, sweep, seed, d0, d1)
        same = ((zg[tb:te] == zo[tb:te]) & (rg[tb:te] == ro[tb:te]) &
                (sg[tb:te] == so[tb:te]))
        say(f"    {int((~same).sum())} of {te - tb} differ")
        assert same.mean() >= parity.MATCH_FRAC, same.mean()
    del zo, ro, so

    say("  whole sweep: update and repair of all tokens")
    s.sweep(sweep, seed)
    zs, rs = s.assignments()
    ss = s.slots()
    c2 = m.rebuild(zg, rg, sg, c)
    promoted = m.repair(zg, rg, sg, c2)
    changed, repaired = s.stats()
    say(f"  promoted {promoted} (library {repaired}), changed {changed}")
    assert repaired == promoted
    assert np.array_equal(zs, zg) and np.array_equal(rs, rg) and np.array_equal(ss, sg)
    N, T, B, Bk = s.totals()
    assert np.array_equal(N, c2.Ngk) and np.array_equal(T, c2.Tgk)
    assert np.array_equal(B, c2.Bkw.T) and np.array_equal(Bk, c2.Bk)
    s.close()
