"""Pins of the oracle's snapshot sampling step, its repair step and its
held-sums ordered sweep, each by an independent re-walk in numpy.

Snapshot step (readings of the sections "Parallel Word Sampling" and
"Parallelism With Improved Accuracy: Word Order Rearrangement": shared counts
frozen at the sweep start, the document's own doc-topic row live, its tokens
in index order).  For every token of the documents walked, the re-walk
  * evaluates the conditionals with the oracle's per-token weight routine
    (itself pinned to ratios of the exact joint in test_oracle_joint.py) on
    the sweep-start counts -- computed here from their definitions, not by
    the oracle -- and on a document row rebuilt in numpy with the tokens
    before it at their new values and the tokens from it on at their old
    values;
  * takes the uniform from the oracle's Philox stream (pinned to rocRAND's
    engine in test_oracle_philox.py) and draws the first outcome whose
    running sum exceeds u times the total;
and the oracle's trace (weights, uniform, sole-head flag) and new state must
equal the re-walk exactly.

Repair (reading A4): in every cell with customers but no table, the token of
smallest index becomes the head; checked against that rule evaluated in numpy
on random states.

Held-sums ordered sweep (reading X2, the default mode of the asynchronous
ablation): sequential in the visiting order with n, t, B_kw and the document
rows live and the sums N_gk, T_gk, B_k held at their sweep-start values; the
re-walk keeps those counts itself and must reproduce the final state and
counts.

Each pin fails on the planted mistakes of tests/mutants.py listed below it.
"""
import numpy as np
import pytest

import oracle
import synth
from tests import mutants


# --------------------------------------------------------------------------
# counts from their definitions (numpy)
# --------------------------------------------------------------------------
def token_groups(m):
    return np.repeat(m.doc_group, np.diff(m.doc_off)).astype(np.int64)


def counts_np(m, z, r):
    """n, t [G, K, V], N, T [G, K], B [K, V], B_k [K] of the state (z, r)."""
    G, K, V = m.G, m.K, m.V
    g = token_groups(m)
    cell = (g * K + z.astype(np.int64)) * V + m.words
    rr = r.astype(np.int64)
    n = np.bincount(cell, minlength=G * K * V).reshape(G, K, V)
    t = np.bincount(cell, weights=rr, minlength=G * K * V).astype(np.int64).reshape(G, K, V)
    return n, t, n.sum(axis=2), t.sum(axis=2), t.sum(axis=0), t.sum(axis=(0, 2))


def as_counts(m, arrays):
    c = m.new_counts()
    n, t, N, T, B, Bk = arrays
    c.n[...], c.t[...], c.Ngk[...], c.Tgk[...], c.Bkw[...], c.Bk[...] = n, t, N, T, B, Bk
    return c


def assert_counts(c, arrays, what):
    for name, want in zip(("n", "t", "Ngk", "Tgk", "Bkw", "Bk"), arrays):
        assert np.array_equal(getattr(c, name), want), f"{what}: {name} differs"


def first_above(w, u):
    """First outcome whose running sum exceeds u times the total (running sums
    in index order, as the draw defines them)."""
    cs = np.cumsum(w)
    return int(np.argmax(cs > u * cs[-1]))


# --------------------------------------------------------------------------
# corpora and states
# --------------------------------------------------------------------------
def make_model(docs, K, V, G, alpha=0.3, a=0.5, b=2.0, gamma=0.1):
    words = np.array([w for _, d in docs for w in d], np.int32)
    doc_off = np.cumsum([0] + [len(d) for _, d in docs]).astype(np.int64)
    doc_group = np.array([g for g, _ in docs], np.int32)
    return oracle.Model(words, doc_off, doc_group, G, K, V, alpha, a, b, gamma)


def repeat_model():
    """Documents that repeat one word many times, so that the tokens of one
    document share count cells and the snapshot/live distinction shows
    within a document; an empty document; a one-token document."""
    docs = [(0, [0] * 30 + [1] * 6 + [0] * 4), (1, [0] * 12 + [2] * 3), (0, []), (1, [1]),
            (0, [2, 0, 2, 0, 2, 0, 1, 1, 1])]
    return make_model(docs, K=3, V=3, G=2, alpha=0.2, a=0.6, b=1.5, gamma=0.3)


def workload_model(idx):
    wl = synth.workload(idx)
    cp = synth.generate(wl, 0)
    return oracle.Model(cp.words, cp.doc_off, cp.doc_group, cp.n_groups, wl.K, wl.vocab,
                        wl.alpha, wl.a, wl.b, wl.gamma)


def evolved_state(m, seed, sweeps):
    """A state after a few snapshot sweeps from the Philox start (the walks
    below then see repeated topics, heads and sole heads)."""
    z, r, c = m.initial_state(seed)
    for s in range(sweeps):
        m.sweep(c, z, r, s, seed + 17, mode="snapshot")
    return z, r


# --------------------------------------------------------------------------
# snapshot step
# --------------------------------------------------------------------------
def check_snapshot_walk(m, z0, r0, sweep, seed, d0=0, d1=None):
    """The oracle's sampling step over documents [d0, d1) against the
    re-walk; returns (tokens walked, sole-head tokens, documents whose row
    changed mid-document)."""
    d1 = m.D if d1 is None else d1
    start = counts_np(m, z0, r0)
    snap = as_counts(m, start)          # what the re-walk reads
    given = as_counts(m, start)         # what the oracle is handed
    z, r = z0.copy(), r0.copy()
    tb, te = int(m.doc_off[d0]), int(m.doc_off[d1])
    _, tw, tu, ts = m.sample_docs(given, z, r, sweep, seed, d0, d1, trace=(tb, te))
    walked = sole = moved_docs = 0
    for d in range(d0, d1):
        b, e = int(m.doc_off[d]), int(m.doc_off[d + 1])
        g = int(m.doc_group[d])
        row = np.bincount(z0[b:e], minlength=m.K).astype(np.int32)
        moved = False
        for i in range(b, e):
            # the document row seen by token i: tokens < i new, tokens >= i old
            want_row = (np.bincount(np.concatenate([z[b:i], z0[i:e]]), minlength=m.K)
                        .astype(np.int32))
            assert np.array_equal(row, want_row)
            w = m.token_weights(snap, row, g, int(m.words[i]), int(z0[i]), int(r0[i]))
            walked += 1
            if w is None:
                sole += 1
                assert ts[i - tb] == 1, f"token {i}: sole head not flagged"
                assert z[i] == z0[i] and r[i] == r0[i], f"token {i}: sole head moved"
                continue
            assert ts[i - tb] == 0, f"token {i}: flagged as sole head"
            assert np.array_equal(tw[i - tb], w), f"token {i}: weights differ from the re-walk"
            u = oracle.uniform(seed, i, sweep)
            assert tu[i - tb] == u, f"token {i}: uniform differs"
            j = first_above(w, u)
            k1, r1 = j // 2, 1 - j % 2
            assert (z[i], r[i]) == (k1, r1), f"token {i}: drew {(z[i], r[i])}, re-walk {(k1, r1)}"
            moved |= k1 != z0[i]
            row[z0[i]] -= 1
            row[k1] += 1
        moved_docs += moved
    # the counts handed to the step are read only
    assert_counts(given, start, "sampling step changed its snapshot")
    return walked, sole, moved_docs


@pytest.mark.parametrize("sweeps,sweep,seed", [(0, 0, 11), (3, 3, 5), (7, 7, 123)])
def test_snapshot_step_repeat_corpus(sweeps, sweep, seed):
    m = repeat_model()
    z0, r0 = evolved_state(m, seed, sweeps)
    walked, sole, moved = check_snapshot_walk(m, z0, r0, sweep, seed)
    assert walked == m.N and moved >= 1


@pytest.mark.parametrize("idx,d1,sweeps", [(0, None, 3), (1, 150, 2)])
def test_snapshot_step_workloads(idx, d1, sweeps):
    m = workload_model(idx)
    z0, r0 = evolved_state(m, 7, sweeps)
    walked, sole, moved = check_snapshot_walk(m, z0, r0, sweeps, 2024, 0, d1)
    assert moved >= 10 and sole >= 1, (walked, sole, moved)


def test_snapshot_step_sole_heads_present():
    """The repeat corpus reaches states with sole heads (the point-mass rule
    is exercised by the walk, not only the draw)."""
    m = repeat_model()
    total_sole = 0
    for s in range(6):
        z0, r0 = evolved_state(m, 3, s)
        total_sole += check_snapshot_walk(m, z0, r0, s, 99)[1]
    assert total_sole >= 1


_LIVE_MOVE = (
    "{ or_counts *cs = (or_counts *)s; const int64_t Vv = m->vocab, wv = m->words[i];"
    " const int64_t c0 = ((int64_t)g * K + k0) * Vv + wv, c1 = ((int64_t)g * K + k1) * Vv + wv;"
    " cs->n[c0] -= 1; cs->Ngk[(int64_t)g * K + k0] -= 1;"
    " if (r0) { cs->t[c0] -= 1; cs->Tgk[(int64_t)g * K + k0] -= 1; cs->Bkw[k0 * Vv + wv] -= 1;"
    " cs->Bk[k0] -= 1; }"
    " cs->n[c1] += 1; cs->Ngk[(int64_t)g * K + k1] += 1;"
    " if (r1) { cs->t[c1] += 1; cs->Tgk[(int64_t)g * K + k1] += 1; cs->Bkw[k1 * Vv + wv] += 1;"
    " cs->Bk[k1] += 1; } }"
)

SNAPSHOT_MUTANTS = {
    # the document row is not kept live: later tokens see the sweep-start row
    "row_not_live": ("or_sample_docs", "crow[k0] -= 1;\n                crow[k1] += 1;", ""),
    # the shared counts are updated live during the step (the sequential
    # sampler's bookkeeping) instead of staying at their sweep-start values
    "live_shared_counts": ("or_sample_docs", "z[i] = k1;", _LIVE_MOVE + " z[i] = k1;"),
    # the removal ignores the stored r (every token leaves as a non-head)
    "removal_ignores_r": ("or_token_weights", "const int64_t tw = s->t[cell] - del * r0;",
                          "const int64_t tw = s->t[cell];"),
    # the draw takes the outcome before the crossing
    "draw_off_by_one": ("draw_outcome", "if (acc > target) return (int)j;",
                        "if (acc > target) return (int)(j > 0 ? j - 1 : 0);"),
}


def caught_by(mutant, check):
    """Run check() (an assertion-based pin) on the oracle built from a mutant,
    on one thread; True if it fails."""
    fn, old, new = mutant
    with mutants.Mutant(fn, old, new) as mut:
        threads = oracle.num_threads()
        oracle.set_num_threads(1)
        try:
            with oracle.swap_library(mut.path):
                try:
                    check()
                except AssertionError:
                    return True
        finally:
            oracle.set_num_threads(threads)
    return False


@pytest.mark.parametrize("name", sorted(SNAPSHOT_MUTANTS))
def test_snapshot_pin_catches_mutant(name):
    m = repeat_model()
    z0, r0 = evolved_state(m, 5, 3)

    def check():
        for sweep in range(3, 9):
            check_snapshot_walk(m, z0, r0, sweep, 41)

    assert caught_by(SNAPSHOT_MUTANTS[name], check), f"snapshot pin misses mutant {name}"


# --------------------------------------------------------------------------
# repair
# --------------------------------------------------------------------------
def check_repair(m, z, r):
    """The oracle's repair of (z, r) against the rule evaluated in numpy;
    returns the number of heads promoted."""
    G, K, V = m.G, m.K, m.V
    cell = (token_groups(m) * K + z.astype(np.int64)) * V + m.words
    n = np.bincount(cell, minlength=G * K * V)
    t = np.bincount(cell, weights=r.astype(np.int64), minlength=G * K * V)
    need = np.flatnonzero((n > 0) & (t == 0))
    first = np.full(G * K * V, m.N, dtype=np.int64)
    np.minimum.at(first, cell, np.arange(m.N))
    r_want = r.copy()
    r_want[first[need]] = 1
    c = m.rebuild(z, r)
    rr = r.copy()
    promoted = m.repair(z, rr, c)
    assert promoted == need.size, f"promoted {promoted}, rule {need.size}"
    assert np.array_equal(rr, r_want), "repair promoted other tokens than the rule"
    assert_counts(c, counts_np(m, z, r_want), "counts after repair")
    return promoted


def random_states(m, seed, n):
    rng = np.random.default_rng(seed)
    for case in range(n):
        z = rng.integers(0, m.K, size=m.N).astype(np.int32)
        p1 = (0.0, 0.05, 0.3, 0.7)[case % 4]
        r = (rng.random(m.N) < p1).astype(np.uint8)
        yield z, r


@pytest.mark.parametrize("idx", [None, 0, 1])
def test_repair_matches_rule(idx):
    m = repeat_model() if idx is None else workload_model(idx)
    total = 0
    for z, r in random_states(m, 3 if idx is None else idx, 8):
        total += check_repair(m, z, r)
    assert total > 0


REPAIR_MUTANTS = {
    # the promoted head's table is not counted, so a second r = 0 token of
    # the same cell is promoted too
    "cell_t_not_updated": ("or_repair", "c->t[(g * K + k) * V + w] += 1;", ""),
    # the promoted head's table is missing from the shadow base
    "base_not_updated": ("or_repair", "c->Bkw[k * V + w] += 1;", ""),
    # the last (largest-index) r = 0 token of the cell is promoted
    "last_token_promoted": (
        "or_repair", "for (int64_t i = m->doc_off[d]; i < m->doc_off[d + 1]; ++i) {",
        "for (int64_t i = m->doc_off[d + 1] - 1; i >= m->doc_off[d]; --i) {"),
}


@pytest.mark.parametrize("name", sorted(REPAIR_MUTANTS))
def test_repair_pin_catches_mutant(name):
    m = repeat_model()

    def check():
        for z, r in random_states(m, 3, 8):
            check_repair(m, z, r)

    assert caught_by(REPAIR_MUTANTS[name], check), f"repair pin misses mutant {name}"


# --------------------------------------------------------------------------
# held-sums ordered sweep
# --------------------------------------------------------------------------
def walk_ordered(m, z0, r0, order, sweep, seed, held):
    """Sequential sweep in the visiting order, re-walked: n, t, B_kw and the
    document rows live; the sums held at their sweep-start values if `held`.
    Returns the final (z, r)."""
    K, V = m.K, m.V
    start = counts_np(m, z0, r0)
    view = as_counts(m, start)     # the counts the conditionals read
    z, r = z0.copy(), r0.copy()
    tok_doc = np.repeat(np.arange(m.D), np.diff(m.doc_off))
    rows = np.zeros((m.D, K), np.int32)
    np.add.at(rows, (tok_doc, z0), 1)
    for i in order:
        d = tok_doc[i]
        g, w, k0, r0i = int(m.doc_group[d]), int(m.words[i]), int(z[i]), int(r[i])
        wts = m.token_weights(view, rows[d], g, w, k0, r0i)
        if wts is None:
            continue
        j = first_above(wts, oracle.uniform(seed, int(i), sweep))
        k1, r1 = j // 2, 1 - j % 2
        for k, rr, sgn in ((k0, r0i, -1), (k1, r1, +1)):
            view.n[g, k, w] += sgn
            if not held:
                view.Ngk[g, k] += sgn
            if rr:
                view.t[g, k, w] += sgn
                view.Bkw[k, w] += sgn
                if not held:
                    view.Tgk[g, k] += sgn
                    view.Bk[k] += sgn
        rows[d, k0] -= 1
        rows[d, k1] += 1
        z[i], r[i] = k1, r1
    return z, r


def check_ordered(m, z0, r0, sweep, seed, held, order=None):
    order = m.interleaved_order() if order is None else order
    zw, rw = walk_ordered(m, z0, r0, order, sweep, seed, held)
    z, r = z0.copy(), r0.copy()
    c = as_counts(m, counts_np(m, z0, r0))
    m.sweep(c, z, r, sweep, seed, mode="ordered", order=order, stale_totals=held)
    assert np.array_equal(z, zw) and np.array_equal(r, rw), "ordered sweep differs from re-walk"
    # the sweep leaves every count live and exact
    assert_counts(c, counts_np(m, z, r), "counts after the ordered sweep")
    return int(np.sum(z != z0))


@pytest.mark.parametrize("held", [True, False])
@pytest.mark.parametrize("idx", [None, 0])
def test_ordered_sweep_matches_rewalk(idx, held):
    m = repeat_model() if idx is None else workload_model(idx)
    moved = 0
    for s in range(3):
        z0, r0 = evolved_state(m, 9, s)
        moved += check_ordered(m, z0, r0, s, 77, held)
    assert moved > 0


ORDERED_MUTANTS = {
    # the sums are not held (the held-sums view is never installed)
    "sums_not_held": ("or_sweep_ordered", "view.Ngk = frozen;", ""),
    # the document row is not kept live
    "row_not_live": ("or_sweep_ordered", "crow[k0] -= 1;\n        crow[k1] += 1;", ""),
    # the token is not removed from its old cell
    "no_removal": ("or_sweep_ordered", "apply_token(m, c, g, wd, k0, r0, -1);", ""),
}


@pytest.mark.parametrize("name", sorted(ORDERED_MUTANTS))
def test_ordered_pin_catches_mutant(name):
    m = repeat_model()

    def check():
        for s in range(4):
            z0, r0 = evolved_state(m, 9, s)
            check_ordered(m, z0, r0, s, 77, True)

    assert caught_by(ORDERED_MUTANTS[name], check), f"ordered-sweep pin misses mutant {name}"
