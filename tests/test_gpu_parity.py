"""GPU parity: the HIP library against the fp64 oracle, through the C ABI.

Each test prints the case it runs before touching the GPU.
"""
import numpy as np
import pytest

import oracle
import synth
from tests import parity

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)


@pytest.fixture(scope="module")
def corpora():
    return {i: synth.generate(synth.workload(i), 0) for i in (0, 1, 2)}


@pytest.mark.parametrize("idx", [0, 1, 2])
def test_initial_state_bit_exact(corpora, idx):
    wl = synth.workload(idx)
    say(f"initial state, workload {wl.name}")
    cp = corpora[idx]
    s, m = parity.make_pair(cp, wl, init_seed=5)
    z0, r0, c0 = m.initial_state(5)
    zg, rg = s.assignments()
    assert np.array_equal(zg, z0)
    assert np.array_equal(rg, r0)
    parity.assert_counts_equal(s, c0)
    s.close()


@pytest.mark.parametrize("idx,sweeps", [(0, 12), (1, 6), (2, 2)])
def test_sweeps_parity(corpora, idx, sweeps):
    wl = synth.workload(idx)
    cp = corpora[idx]
    s, m = parity.make_pair(cp, wl, init_seed=1)
    for sw in range(sweeps):
        say(f"sweep parity, workload {wl.name}, sweep {sw}")
        rep, changed, repaired = parity.one_step(s, m, sw, seed=2024 + idx)
        say(f"  {rep} changed={changed} repaired={repaired}")
        assert changed > 0
    s.close()


def test_late_sweeps_parity_g4(corpora):
    """The per-sweep protocol on the 3M-token workload at sweeps 0, 1, 50 and
    99 of a 100-sweep run (the sweeps between run on the library only), with
    the joint compared before each of them and at the end."""
    wl = synth.workload(2)
    cp = corpora[2]
    s, m = parity.make_pair(cp, wl, init_seed=1)
    seed = 2026
    for sw in range(100):
        if sw in (0, 1, 50, 99):
            z, r = s.assignments()
            ll_g, ll_o = s.loglik(), m.loglik(z, r, m.rebuild(z, r))
            say(f"sweep parity, workload {wl.name}, sweep {sw}: joint {ll_g!r} / {ll_o!r}")
            assert abs(ll_g - ll_o) <= parity.LL_RTOL * abs(ll_o)
            rep, changed, repaired = parity.one_step(s, m, sw, seed)
            say(f"  {rep} changed={changed} repaired={repaired}")
        else:
            s.sweep(sw, seed)
    z, r = s.assignments()
    ll_g, ll_o = s.loglik(), m.loglik(z, r, m.rebuild(z, r))
    assert abs(ll_g - ll_o) <= parity.LL_RTOL * abs(ll_o)
    s.close()


@pytest.mark.parametrize("idx", [0, 1, 2])
def test_loglik_parity(corpora, idx):
    wl = synth.workload(idx)
    say(f"loglik parity, workload {wl.name}")
    cp = corpora[idx]
    s, m = parity.make_pair(cp, wl, init_seed=3)
    for sw in range(3):
        z, r = s.assignments()
        c = m.rebuild(z, r)
        ll_o = m.loglik(z, r, c)
        ll_g = s.loglik()
        say(f"  sweep {sw}: gpu {ll_g!r} oracle {ll_o!r}")
        assert abs(ll_g - ll_o) <= parity.LL_RTOL * abs(ll_o)
        s.sweep(sw, 77)
    # generator truth through set_assignments
    s.set_assignments(cp.z_true, cp.r_true)
    zt, rt = cp.z_true.copy(), cp.r_true.copy()
    ct = m.rebuild(zt, rt)
    assert abs(s.loglik() - m.loglik(zt, rt, ct)) <= 1e-6 * abs(m.loglik(zt, rt, ct))
    s.close()


def test_determinism_and_resume(corpora):
    wl = synth.workload(1)
    say(f"determinism and resume, workload {wl.name}")
    cp = corpora[1]
    a, _ = parity.make_pair(cp, wl, init_seed=9)
    b, _ = parity.make_pair(cp, wl, init_seed=9)
    for sw in range(3):
        a.sweep(sw, 55)
        b.sweep(sw, 55)
    za, ra = a.assignments()
    zb, rb = b.assignments()
    assert np.array_equal(za, zb) and np.array_equal(ra, rb)
    # checkpoint a, continue both; resume a fresh state from the checkpoint
    c, _ = parity.make_pair(cp, wl, init_seed=123)
    c.set_assignments(za, ra)
    for sw in range(3, 6):
        a.sweep(sw, 55)
        c.sweep(sw, 55)
    za, ra = a.assignments()
    zc, rc = c.assignments()
    assert np.array_equal(za, zc) and np.array_equal(ra, rc)
    na, ta = a.counts()
    nc, tc = c.counts()
    assert np.array_equal(na, nc) and np.array_equal(ta, tc)
    for x in (a, b, c):
        x.close()


def test_debug_hook_is_repeatable(corpora):
    wl = synth.workload(0)
    say("same sampling step twice from an identical state")
    cp = corpora[0]
    s, _ = parity.make_pair(cp, wl, init_seed=4)
    z, r = s.assignments()
    w1, u1, zr1 = s.conditionals(0, 1, 0, s.N)
    w2, u2, zr2 = s.conditionals(0, 1, 0, s.N)
    assert np.array_equal(zr1, zr2) and np.array_equal(w1, w2)
    s.close()


def test_repair_from_all_r_zero(corpora):
    wl = synth.workload(1)
    say(f"repair path, workload {wl.name}")
    cp = corpora[1]
    s, m = parity.make_pair(cp, wl, init_seed=0)
    rng = np.random.default_rng(0)
    for case in ("all_zero", "random"):
        z = rng.integers(0, wl.K, size=cp.n_tokens).astype(np.int32)
        r = (np.zeros(cp.n_tokens, np.uint8) if case == "all_zero"
             else rng.integers(0, 2, size=cp.n_tokens).astype(np.uint8))
        s.set_assignments(z, r)
        zo, ro = z.copy(), r.copy()
        c = m.rebuild(zo, ro)
        m.repair(zo, ro, c)
        zg, rg = s.assignments()
        assert np.array_equal(zg, zo) and np.array_equal(rg, ro), case
        parity.assert_counts_equal(s, c)
    s.close()


def test_bad_assignments_rejected(corpora):
    from paper_1510_06549_amd import spdp as sp

    wl = synth.workload(0)
    say("invalid assignments are rejected")
    cp = corpora[0]
    s, _ = parity.make_pair(cp, wl)
    z = np.zeros(cp.n_tokens, np.int32)
    z[5] = wl.K  # out of range
    with pytest.raises(sp.SpdpError) as e:
        s.set_assignments(z, np.zeros(cp.n_tokens, np.uint8))
    assert e.value.code == sp.SPDP_E_ARG
    s.close()
