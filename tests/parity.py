"""Helpers of the GPU-vs-oracle parity tests (no tests in this module).

The comparison protocol, per sweep, from one identical state:
  (i)   counts: the library's counts equal the oracle's rebuild of the
        library's (z, r), bit for bit;
  (ii)  conditionals: the library's fp32 weights equal the oracle's fp64 ones
        within 1e-5 relative (exact zeros where the oracle has zeros), for
        tokens whose earlier same-document tokens were sampled identically;
  (iii) samples: (z, r) identical on >= 99.99% of tokens, and every first
        mismatch of a document has its uniform within 1e-5 of the oracle's
        normalised CDF boundary between the two outcomes;
  (iv)  after update and repair the library's state and counts equal the
        oracle's rebuild and repair of the library's sampled (z, r).
With word associations the state is (z, r, source slot), the outcomes per
token are K (S + 1) and every token draws (the sole head redraws its source).
"""
from __future__ import annotations

import dataclasses

import numpy as np

import oracle
from paper_1510_06549_amd import spdp as sp

W_RTOL = 1e-5
U_TOL = 1e-5
LL_RTOL = 1e-6
MATCH_FRAC = 0.9999


def make_pair(cp, wl, init_seed=0, K=None, assoc=None):
    """Library state and oracle model of one corpus; assoc = (row_off, src, p)
    for the model with word associations."""
    K = wl.K if K is None else K
    s = sp.Sampler(cp.words, cp.doc_off, cp.doc_group, cp.n_groups, cp.vocab, K, wl.alpha, wl.a,
                   wl.b, wl.gamma, init_seed=init_seed, assoc=assoc)
    args = (cp.words, cp.doc_off, cp.doc_group, cp.n_groups, K, cp.vocab, wl.alpha, wl.a, wl.b,
            wl.gamma)
    m = oracle.Model(*args) if assoc is None else oracle.AssocModel(*args, *assoc)
    return s, m


def _is_assoc(m) -> bool:
    return isinstance(m, oracle.AssocModel)


def state_of(s: sp.Sampler, m):
    """The library's current state as the oracle takes it: (z, r) or (z, r, slot)."""
    z, r = s.assignments()
    return (z, r, s.slots()) if _is_assoc(m) else (z, r)


def unpack(zr):
    """Packed sampled outcomes -> (z, r, slot)."""
    return (zr & 0xFFFF) >> 1, (zr & 1).astype(np.uint8), (zr >> 16).astype(np.uint8)


def assert_counts_equal(s: sp.Sampler, c: oracle.Counts):
    n, t = s.counts()
    assert np.array_equal(n, c.n), "customer counts differ"
    assert np.array_equal(t, c.t), "table counts differ"
    N, T, B, Bk = s.totals()
    assert np.array_equal(N, c.Ngk), "N_gk differs"
    assert np.array_equal(T, c.Tgk), "T_gk differs"
    assert np.array_equal(B, c.Bkw.T), "B differs"
    assert np.array_equal(Bk, c.Bk), "B_k differs"


@dataclasses.dataclass
class StepReport:
    n_tokens: int
    mismatches: int
    primary: int
    max_primary_gap: float
    max_w_rel: float
    weights_checked: int


def _chunks(m, chunk_tokens):
    d = 0
    off = m.doc_off
    while d < m.D:
        d_end = int(np.searchsorted(off, off[d] + chunk_tokens, side="left"))
        d_end = min(max(d_end, d + 1), m.D)
        yield d, d_end, int(off[d]), int(off[d_end])
        d = d_end


def _outcome(m, z, r, sl):
    """Index of the outcome (z, r[, slot]) in the token's weight vector."""
    if _is_assoc(m):
        return (m.S + 1) * int(z) + (int(sl) if r else m.S)
    return 2 * int(z) + (1 - int(r))


def one_step(s: sp.Sampler, m: oracle.Model, sweep: int, seed: int, chunk_tokens=150_000):
    """Run one sweep on both sides from the library's current state and compare."""
    assoc = _is_assoc(m)
    st = state_of(s, m)
    c = m.rebuild(*st)
    assert_counts_equal(s, c)  # (i)
    zo, ro = st[0].copy(), st[1].copy()
    so = st[2].copy() if assoc else np.zeros(m.N, np.uint8)
    ost = (zo, ro, so) if assoc else (zo, ro)
    zg_pre = np.empty(m.N, dtype=np.int32)
    rg_pre = np.empty(m.N, dtype=np.uint8)
    sg_pre = np.zeros(m.N, dtype=np.uint8)
    n_mism = primary = checked = 0
    primary_gap = max_rel = 0.0
    for d0, d1, tb, te in _chunks(m, chunk_tokens):
        if te == tb:
            continue
        # library: weights, uniforms and samples of the (uncommitted) sampling step
        w_g, u_g, zr_g = s.conditionals(sweep, seed, tb, te)
        # oracle: the same documents with a full trace
        _, w_o, u_o, skip_o = m.sample_docs(c, *ost, sweep, seed, d0, d1, trace=(tb, te))
        skip_o = skip_o.astype(bool)
        zg, rg, sg = unpack(zr_g)
        zg_pre[tb:te], rg_pre[tb:te], sg_pre[tb:te] = zg, rg, sg
        if not assoc:
            assert not sg.any(), "slot bits in a state without associations"

        # (iii) samples
        same = (zg == zo[tb:te]) & (rg == ro[tb:te]) & (sg == so[tb:te])
        mism = np.flatnonzero(~same)
        n_mism += len(mism)
        doc = np.repeat(np.arange(d0, d1), np.diff(m.doc_off[d0:d1 + 1])) - d0
        first_bad = np.full(d1 - d0, np.iinfo(np.int64).max, dtype=np.int64)
        if len(mism):
            np.minimum.at(first_bad, doc[mism], mism)
        for i in np.unique(first_bad[first_bad < np.iinfo(np.int64).max]):
            primary += 1
            assert not skip_o[i], f"token {tb + i}: oracle kept it (sole head), library moved it"
            jg = _outcome(m, zg[i], rg[i], sg[i])
            jo = _outcome(m, zo[tb + i], ro[tb + i], so[tb + i])
            cdf = np.cumsum(w_o[i])
            cdf /= cdf[-1]
            gap = abs(u_o[i] - cdf[min(jg, jo)])
            primary_gap = max(primary_gap, gap)
            assert gap <= U_TOL, f"token {tb + i}: u={u_o[i]} boundary={cdf[min(jg, jo)]}"

        # (ii) conditionals, for tokens up to their document's first mismatch
        ok_tok = np.arange(te - tb) <= first_bad[doc]
        assert np.array_equal((u_g < 0)[ok_tok], skip_o[ok_tok]), "sole-head rule differs"
        sel = ok_tok & ~skip_o
        wg = w_g[sel].astype(np.float64)
        wo = w_o[sel]
        zero_o = wo == 0.0
        assert np.all(wg[zero_o] == 0.0), "library weight nonzero where the oracle has zero"
        rel = np.abs(wg[~zero_o] - wo[~zero_o]) / wo[~zero_o]
        if rel.size:
            max_rel = max(max_rel, float(rel.max()))
        assert max_rel <= W_RTOL, f"weight relative error {max_rel}"
        assert np.array_equal(u_g[sel].astype(np.float64), u_o[sel]), "uniforms differ"
        checked += int(sel.sum())
    frac = 1.0 - n_mism / max(m.N, 1)
    assert frac >= MATCH_FRAC, f"only {frac:.6f} of tokens agree"

    # commit the library's sweep
    s.sweep(sweep, seed)
    st2 = state_of(s, m)
    # (iv) update + repair: oracle rebuild and repair of the library's samples
    pre = (zg_pre, rg_pre, sg_pre) if assoc else (zg_pre, rg_pre)
    c2 = m.rebuild(*pre)
    m.repair(*pre, c2)
    for a, b in zip(st2, pre):
        assert np.array_equal(a, b), "post-repair state differs"
    assert_counts_equal(s, c2)
    changed, repaired = s.stats()
    return StepReport(m.N, n_mism, primary, primary_gap, max_rel, checked), changed, repaired
