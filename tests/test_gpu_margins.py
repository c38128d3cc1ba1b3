"""The fp32 sampling path against the rounding bound that its fp64 re-decision
margin rests on, through the C ABI.

The samplers take a draw again in fp64 when the target lies within
(4 KPL + 32) 2^-24 of the total from a CDF boundary (plain model) or
(4 KPL + SP + 32) 2^-24 (word associations).  The bound behind those margins
counts at most 9 roundings in a plain fp32 weight (alpha, gamma, the per-topic
constant and the ratio pair rounded once each from fp64, two sums with counts,
three products); a traced association weight, formed as hq (p bv), carries at
most 11.  Checked here, over several sweeps of three corpora, each plain and
with word associations:
  (a) every traced fp32 weight is within that many roundings of the oracle's
      fp64 weight (relative);
  (b) no token's sample differs from the oracle's: a margin below the sampler's
      real error would let some decision near a boundary come out differently.
Each test prints the case it runs before touching the GPU.
"""
import pytest

import synth
from tests import parity

pytestmark = pytest.mark.gpu

U = 2.0 ** -24
PLAIN_WEIGHT_ROUNDINGS = 9
ASSOC_WEIGHT_ROUNDINGS = 11


def say(*a):
    print(*a, flush=True)


def _run(idx, sweeps, roundings, assoc_sources=0):
    wl = synth.workload(idx)
    cp = synth.generate(wl, 0)
    assoc = (synth.associations(cp.n_groups, cp.vocab, assoc_sources, 0.3, 5)
             if assoc_sources else None)
    s, m = parity.make_pair(cp, wl, init_seed=3, assoc=assoc)
    worst = 0.0
    for sw in range(sweeps):
        say(f"margins, workload {wl.name}, sources {assoc_sources}, sweep {sw}")
        rep, changed, _ = parity.one_step(s, m, sw, seed=77 + idx)
        say(f"  {rep}")
        assert rep.mismatches == 0, f"{rep.mismatches} samples differ from the oracle"
        worst = max(worst, rep.max_w_rel)
        assert changed > 0
    s.close()
    say(f"  largest relative weight error {worst:.3e} = {worst / U:.2f} u")
    # first order in u; the second-order term is below 1e-6 of the bound
    assert worst <= roundings * U * (1.0 + 1e-6)


@pytest.mark.parametrize("idx,sweeps", [(0, 6), (1, 3), (2, 1)])
def test_plain_weights_within_bound_and_draws_exact(idx, sweeps):
    _run(idx, sweeps, PLAIN_WEIGHT_ROUNDINGS)


@pytest.mark.parametrize("idx,sweeps,sources", [(0, 6, 2), (1, 3, 4), (2, 1, 4)])
def test_assoc_weights_within_bound_and_draws_exact(idx, sweeps, sources):
    _run(idx, sweeps, ASSOC_WEIGHT_ROUNDINGS, sources)
