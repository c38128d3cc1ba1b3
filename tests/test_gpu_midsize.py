"""Parity at the 40M-token workload (10 groups x 20 000 documents, K = 200),
where the oracle can sample the whole sweep in test time:
  * counts: totals, shadow base and two whole groups' count rows of the
    library's state equal the oracle's rebuild, bit for bit;
  * sampling: every token's sampled (z, r) equals the oracle's sampling step
    on the same state, seed and sweep (>= 99.99 % required; identical in
    practice), and for documents at the start, middle and end of the corpus
    the weights and uniforms are compared one by one;
  * update and repair: the library's state and totals after the sweep equal
    the oracle's rebuild and repair of the library's sampled state.
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


@pytest.mark.parametrize("warm,seed", [(1, 4321), (25, 1000)])
def test_midsize_workload_every_draw(warm, seed):
    """warm = 1: the sweep after one warm-up sweep; warm = 25: the sweep after
    the benchmark's schedule of 5 warm-up and 20 timed sweeps (its seed).
    The joint (Eq. SPDP-Blocked-Gibbs-Joint-Prob, P = I) is compared before
    and after the compared sweep."""
    import torch

    wl = synth.workload("g10-d20000-k200")
    say(f"mid-size parity, workload {wl.name}, after {warm} sweep(s): generating corpus")
    cp = synth.generate(wl, 0)
    s = parity.sp.Sampler(cp.words, cp.doc_off, cp.doc_group, cp.n_groups, wl.vocab, wl.K,
                          wl.alpha, wl.a, wl.b, wl.gamma, init_seed=0,
                          hip_stream=torch.cuda.current_stream().cuda_stream)
    say(f"  {warm} warm-up sweep(s)")
    for sw in range(warm):
        s.sweep(sw, seed)
    z, r = s.assignments()
    say("  oracle model and dense rebuild")
    m = oracle.Model(cp.words, cp.doc_off, cp.doc_group, cp.n_groups, wl.K, wl.vocab, wl.alpha,
                     wl.a, wl.b, wl.gamma)
    c = m.rebuild(z, r)
    assert m.repair(z.copy(), r.copy(), c.copy()) == 0, "library state has a cell without a head"

    say("  counts")
    N, T, B, Bk = s.totals()
    assert np.array_equal(N, c.Ngk) and np.array_equal(T, c.Tgk)
    assert np.array_equal(B, c.Bkw.T) and np.array_equal(Bk, c.Bk)
    for g in (0, cp.n_groups - 1):
        n_g, t_g = s.counts(g, g + 1)
        assert np.array_equal(n_g[0], c.n[g]), f"n of group {g}"
        assert np.array_equal(t_g[0], c.t[g]), f"t of group {g}"
    del n_g, t_g
    ll_g, ll_o = s.loglik(), m.loglik(z, r, c)
    say(f"  joint: library {ll_g!r} oracle {ll_o!r}")
    assert abs(ll_g - ll_o) <= parity.LL_RTOL * abs(ll_o)

    sweep = warm
    say("  every token: library draws vs the oracle's sampling step")
    zr_pre = s.sampled(sweep, seed)
    zg, rg = (zr_pre >> 1).astype(np.int32), (zr_pre & 1).astype(np.uint8)
    zo, ro = z.copy(), r.copy()
    m.sample_docs(c, zo, ro, sweep, seed)
    same = (zg == zo) & (rg == ro)
    say(f"  {int((~same).sum())} of {m.N} draws differ")
    assert same.mean() >= parity.MATCH_FRAC, same.mean()

    for d0 in (0, m.D // 2 + 11, m.D - 200):
        d1 = d0 + 200
        tb, te = int(m.doc_off[d0]), int(m.doc_off[d1])
        say(f"  documents [{d0}, {d1}): weights and uniforms of tokens [{tb}, {te})")
        w_g, u_g, _ = s.conditionals(sweep, seed, tb, te)
        zt, rt = z.copy(), r.copy()
        _, w_o, u_o, skip_o = m.sample_docs(c, zt, rt, sweep, seed, d0, d1, trace=(tb, te))
        skip_o = skip_o.astype(bool)
        assert np.array_equal(u_g < 0, skip_o)
        doc = np.repeat(np.arange(d1 - d0), np.diff(m.doc_off[d0:d1 + 1]))
        ok = ~skip_o
        for i in np.flatnonzero(~same[tb:te]):
            ok &= ~((doc == doc[i]) & (np.arange(te - tb) > i))
        wo, wgt = w_o[ok], w_g[ok].astype(np.float64)
        nz = wo != 0
        assert np.all(wgt[~nz] == 0)
        assert np.max(np.abs(wgt[nz] - wo[nz]) / wo[nz]) <= parity.W_RTOL
        assert np.array_equal(u_g[ok].astype(np.float64), u_o[ok])
        del w_g, w_o

    say("  whole sweep: update and repair of all tokens")
    s.sweep(sweep, seed)
    zs, rs = s.assignments()
    c2 = m.rebuild(zg, rg, c)
    promoted = m.repair(zg, rg, c2)
    changed, repaired = s.stats()
    say(f"  promoted {promoted} (library {repaired}), changed {changed}")
    assert repaired == promoted
    assert np.array_equal(zs, zg) and np.array_equal(rs, rg)
    N, T, B, Bk = s.totals()
    assert np.array_equal(N, c2.Ngk) and np.array_equal(T, c2.Tgk)
    assert np.array_equal(B, c2.Bkw.T) and np.array_equal(Bk, c2.Bk)
    ll_g, ll_o = s.loglik(), m.loglik(zs, rs, c2)
    say(f"  joint after the sweep: library {ll_g!r} oracle {ll_o!r}")
    assert abs(ll_g - ll_o) <= parity.LL_RTOL * abs(ll_o)
    s.close()
