"""The invariant checker (spdp_check) on the GPU: silent on every state the
library produces (after creation, sweeps, resume, the asynchronous sweep and
with word associations), and reports SPDP_E_STATE once a single stored count
is corrupted through the debug hook, in each way a count can go wrong (a
customer too many, a table too many, a table in an empty cell); a rebuild
from the state restores it.  Each test prints its case before touching the
GPU.
"""
import numpy as np
import pytest

import synth
from paper_1510_06549_amd import spdp as sp
from tests import parity

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)


def corrupted_is_reported(s, g, w, k, dn, dt):
    s.poke(g, w, k, dn, dt)
    with pytest.raises(sp.SpdpError) as e:
        s.check()
    assert e.value.code == sp.SPDP_E_STATE
    assert "inconsistent" in sp.spdp_last_error()
    s.poke(g, w, k, -dn, -dt)
    assert s.check() == 0


@pytest.mark.parametrize("idx,assoc", [(0, False), (1, False), (1, True)])
def test_check_silent_then_reports_corruption(idx, assoc):
    wl = synth.workload(idx)
    say(f"invariant check, workload {wl.name}, associations {assoc}")
    cp = synth.generate(wl, 0)
    A = synth.associations(cp.n_groups, cp.vocab, 3, 0.3, 1) if assoc else None
    s, m = parity.make_pair(cp, wl, init_seed=2, assoc=A)
    assert s.check() == 0
    for sw in range(3):
        s.sweep(sw, 31)
        assert s.check() == 0
    # a non-empty cell and an empty one of group 0
    n, t = s.counts(0, 1)
    k, w = np.argwhere(n[0] > 0)[0]
    ke, we = np.argwhere(n[0] == 0)[0]
    corrupted_is_reported(s, 0, w, k, 1, 0)      # a customer too many
    corrupted_is_reported(s, 0, w, k, 0, 1)      # a table too many (t may exceed n)
    corrupted_is_reported(s, 0, we, ke, 0, 1)    # a table in an empty cell
    # a corruption left in place is removed by a rebuild from the state
    s.poke(0, w, k, 1, 1)
    with pytest.raises(sp.SpdpError):
        s.check()
    st = parity.state_of(s, m)
    if assoc:
        s.set_assignments(st[0], st[1], st[2])
    else:
        s.set_assignments(st[0], st[1])
    assert s.check() == 0
    s.close()


def test_check_after_async_sweep_and_edge_shapes():
    say("invariant check after the asynchronous sweep and on K = 1 and K = 1024")
    wl = synth.workload(0)
    cp = synth.generate(wl, 0)
    s, _ = parity.make_pair(cp, wl, init_seed=3)
    s.sweep_async(0, 5, 0, False)
    assert s.check() == 0
    s.close()
    for K in (1, 1024):
        s, _ = parity.make_pair(cp, wl, init_seed=4, K=K)
        s.sweep(0, 8)
        assert s.check() == 0
        s.close()


def test_poke_rejects_bad_cells():
    wl = synth.workload(0)
    say("debug poke argument errors")
    cp = synth.generate(wl, 0)
    s, _ = parity.make_pair(cp, wl)
    for args in ((wl.n_groups, 0, 0, 1, 0), (0, wl.vocab, 0, 1, 0), (0, 0, wl.K, 1, 0),
                 (0, 0, 0, -70000, 0)):
        with pytest.raises(sp.SpdpError) as e:
            s.poke(*args)
        assert e.value.code == sp.SPDP_E_ARG
    assert s.check() == 0
    s.close()
