"""Held-out fold-in at the largest workload (20 groups x 50 000 documents,
K = 500; the last 10 % of each group's documents held out: 25 M test tokens in
100 000 documents), in the launch configuration `bench.py --heldout` times.

The group estimates come from the oracle (its rebuild and estimates of the
library's trained state); the oracle then folds in:
  * the first 1 000 test documents: the library's topics of those documents,
    from its fold-in of the whole test corpus, equal the oracle's (a test
    document's chain depends only on its own tokens and their indices);
  * every 100th test document (1 000 documents across all groups), as a corpus
    of their own on both sides: topics equal and total log-likelihood to 1e-9.
Each step prints what it runs before touching the GPU.
"""
import numpy as np
import pytest

import oracle
import synth
from tests import parity

pytestmark = pytest.mark.gpu

SWEEPS = 10
SEED = 31


def say(*a):
    print(*a, flush=True)


def _sub(te, docs):
    """The test documents `docs` (increasing) as a corpus of their own."""
    lens = np.diff(te.doc_off)[docs]
    off = np.zeros(docs.size + 1, dtype=np.int64)
    np.cumsum(lens, out=off[1:])
    words = np.concatenate([te.words[te.doc_off[d]:te.doc_off[d + 1]] for d in docs])
    return words.astype(np.int32), off, te.doc_group[docs].astype(np.int32)


def test_foldin_largest_workload():
    import torch

    wl = synth.workload("g20-d50000-k500")
    say(f"full-size fold-in, workload {wl.name}: generating corpus")
    cp = synth.generate(wl, 0)
    tr, te = synth.split_heldout(cp, 0.1)
    del cp
    say(f"  train {tr.n_tokens} tokens, test {te.n_tokens} tokens in {te.n_docs} documents")
    s = parity.sp.Sampler(tr.words, tr.doc_off, tr.doc_group, tr.n_groups, wl.vocab, wl.K,
                          wl.alpha, wl.a, wl.b, wl.gamma, init_seed=0,
                          hip_stream=torch.cuda.current_stream().cuda_stream)
    say("  one training sweep")
    s.sweep(0, 5)
    z, r = s.assignments()

    say("  oracle rebuild and group estimates")
    m = oracle.Model(tr.words, tr.doc_off, tr.doc_group, tr.n_groups, wl.K, wl.vocab, wl.alpha,
                     wl.a, wl.b, wl.gamma)
    c = m.rebuild(z, r)
    _, _, pg = m.estimates(z, c)
    del c, z, r

    say(f"  library fold-in of all {te.n_docs} test documents, {SWEEPS} sweeps")
    _, _, zt = s.heldout(te.words, te.doc_off, te.doc_group, SWEEPS, SEED)

    n_d = 1000
    ntok = int(te.doc_off[n_d])
    say(f"  oracle fold-in of the first {n_d} test documents ({ntok} tokens)")
    _, zo, _ = m.heldout(pg, te.words[:ntok], te.doc_off[:n_d + 1], te.doc_group[:n_d], SWEEPS,
                         SEED)
    same = float(np.mean(zt[:ntok] == zo))
    say(f"    topics equal {same:.6f}")
    assert same >= parity.MATCH_FRAC

    docs = np.arange(0, te.n_docs, 100)
    w, off, grp = _sub(te, docs)
    assert np.unique(grp).size == tr.n_groups
    say(f"  every 100th test document ({docs.size} documents, {w.size} tokens): library and "
        f"oracle")
    ppl, tot, zs = s.heldout(w, off, grp, SWEEPS, SEED)
    tot_o, zso, _ = m.heldout(pg, w, off, grp, SWEEPS, SEED)
    same = float(np.mean(zs == zso))
    say(f"    topics equal {same:.6f}, log-likelihood {tot:.6f} vs {tot_o:.6f}")
    assert same >= parity.MATCH_FRAC
    assert abs(tot - tot_o) <= 1e-9 * abs(tot_o)
    assert abs(ppl - np.exp(-tot_o / w.size)) <= 1e-9 * ppl
    s.close()
