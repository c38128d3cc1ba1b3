"""GPU edge cases: empty and ragged documents, tiny corpora, topic-count
boundaries of the sampler's lane layout, maximum K, a = 0."""
import math

import numpy as np
import pytest

import oracle
import synth
from tests import parity

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)


class W:  # minimal workload stand-in
    def __init__(self, K, alpha=0.1, a=0.5, b=10.0, gamma=0.01):
        self.K, self.alpha, self.a, self.b, self.gamma = K, alpha, a, b, gamma


def corpus_from_docs(docs, vocab):
    words = np.array([w for _, d in docs for w in d], np.int32)
    doc_off = np.cumsum([0] + [len(d) for _, d in docs]).astype(np.int64)
    doc_group = np.array([g for g, _ in docs], np.int32)
    return synth.Corpus(words, doc_off, doc_group, np.zeros_like(words),
                        np.zeros(len(words), np.uint8), int(doc_group.max()) + 1, vocab)


def test_single_token_closed_form():
    say("single-token corpus")
    cp = corpus_from_docs([(0, [3])], vocab=7)
    wl = W(K=4)
    s, m = parity.make_pair(cp, wl)
    w, u, zr = s.conditionals(0, 1, 0, 1)
    np.testing.assert_allclose(w[0, 0::2], wl.alpha / 7, rtol=1e-6)
    assert np.all(w[0, 1::2] == 0)
    assert zr[0] & 1 == 1
    for sw in range(4):
        parity.one_step(s, m, sw, 3)
    s.close()


def test_empty_and_ragged_documents():
    say("empty and ragged documents")
    rng = np.random.default_rng(1)
    docs = []
    for d in range(300):
        L = [0, 1, 2, 63, 64, 65, 127, 128, 129, 200][d % 10] if d % 3 else int(rng.integers(0, 40))
        docs.append((d % 3, list(rng.integers(0, 50, size=L))))
    cp = corpus_from_docs(docs, vocab=50)
    wl = W(K=13)
    s, m = parity.make_pair(cp, wl)
    for sw in range(5):
        rep, ch, rp = parity.one_step(s, m, sw, 11)
        say(f"  {rep}")
    s.close()


@pytest.mark.parametrize("K", [1, 2, 63, 64, 65, 128, 129, 256, 257, 500, 512, 513, 768, 769, 1024])
def test_topic_count_boundaries(K):
    say(f"K = {K}")
    rng = np.random.default_rng(K)
    docs = [(d % 2, list(rng.zipf(1.3, size=int(rng.integers(1, 120))) % 300)) for d in range(120)]
    cp = corpus_from_docs(docs, vocab=300)
    wl = W(K=K, alpha=0.2, a=0.6, b=5.0, gamma=0.05)
    s, m = parity.make_pair(cp, wl)
    for sw in range(3):
        rep, ch, rp = parity.one_step(s, m, sw, 5 + K)
    ll_o = m.loglik(*s.assignments(), m.rebuild(*s.assignments()))
    assert abs(s.loglik() - ll_o) <= 1e-6 * abs(ll_o)
    s.close()


def test_discount_zero_and_large_concentration():
    say("a = 0 (Dirichlet process restaurants)")
    cp = synth.generate(synth.workload(0), 3)
    wl = W(K=10, alpha=0.3, a=0.0, b=200.0, gamma=0.5)
    s, m = parity.make_pair(cp, wl)
    for sw in range(3):
        parity.one_step(s, m, sw, 8)
    s.close()


def test_invalid_arguments():
    from paper_1510_06549_amd import spdp as sp

    say("invalid arguments")
    words = np.array([0, 1, 2], np.int32)
    off = np.array([0, 3], np.int64)
    grp = np.array([0], np.int32)
    bad = [
        dict(K=0), dict(K=2000), dict(alpha=0.0), dict(a=1.0), dict(b=0.0), dict(gamma=-1.0),
    ]
    for kw in bad:
        args = dict(K=4, alpha=0.1, a=0.5, b=1.0, gamma=0.1)
        args.update(kw)
        with pytest.raises(sp.SpdpError) as e:
            sp.spdp_create(words, off, grp, 1, 3, args["K"], args["alpha"], args["a"], args["b"],
                           args["gamma"])
        assert e.value.code == sp.SPDP_E_ARG
    with pytest.raises(sp.SpdpError):  # word id out of range
        sp.spdp_create(np.array([0, 5], np.int32), np.array([0, 2], np.int64), grp, 1, 3, 4, 0.1,
                       0.5, 1.0, 0.1)
    with pytest.raises(sp.SpdpError):  # group out of range
        sp.spdp_create(words, off, np.array([1], np.int32), 1, 3, 4, 0.1, 0.5, 1.0, 0.1)


def test_shadow_base_counts_beyond_16_bits():
    """A shadow-base count above 65535 (the sampler's 32-bit launch then
    reads B itself where the 16-bit copy saturates): 4 groups each with 16400
    occurrences of word 0, all seated at their own table of topic 0, give
    B[0][0] = 65600."""
    say("shadow-base count beyond 16 bits")
    rng = np.random.default_rng(7)
    docs = []
    for g in range(4):
        for _ in range(4):
            d = [0] * 4100 + list(rng.integers(1, 3, size=20))
            rng.shuffle(d)
            docs.append((g, d))
    cp = corpus_from_docs(docs, vocab=3)
    wl = W(K=3, alpha=0.5, a=0.3, b=50.0, gamma=0.1)
    s, m = parity.make_pair(cp, wl)
    z = np.zeros(cp.n_tokens, np.int32)
    r = np.ones(cp.n_tokens, np.uint8)
    s.set_assignments(z, r)
    _, _, B, _ = s.totals()
    assert B[0, 0] == 65600
    rep, ch, rp = parity.one_step(s, m, 0, 21)
    say(f"  {rep}")
    s.close()


def test_shadow_base_beyond_16_bits_with_many_documents():
    """The 32-bit shadow-base launch at 8 topics per lane (K = 500) over 5 000
    documents, more than the workgroups of that launch's persistent grid, so
    that workgroups claim several documents each: 4 groups of 1 250 documents,
    14 occurrences of word 0 in each, all seated at their own table of topic 0
    (B[0][0] = 70 000), and 6 other tokens per document at random states."""
    say("shadow-base count beyond 16 bits, K = 500, 5000 documents")
    wide_base_case(None)


def test_shadow_base_beyond_16_bits_with_word_associations():
    """The association sampler's 32-bit shadow-base launch in the instance the
    benchmark runs (K = 500, four sources per word), over more documents than
    its persistent grid has workgroups: the corpus of the test above, every
    table of word 0 at topic 0 drawing its first source, which is word 0
    itself, so the source-keyed count B[0][0] = 70 000."""
    say("shadow-base count beyond 16 bits, word associations, K = 500")
    wide_base_case(4)


def wide_base_case(sources):
    rng = np.random.default_rng(11)
    V, K = 60, 500
    docs = []
    for g in range(4):
        for _ in range(1250):
            d = [0] * 14 + list(rng.integers(1, V, size=6))
            rng.shuffle(d)
            docs.append((g, d))
    cp = corpus_from_docs(docs, vocab=V)
    wl = W(K=K, alpha=0.1, a=0.4, b=20.0, gamma=0.05)
    assoc = synth.associations(4, V, sources, 0.3, 5) if sources else None
    s, m = parity.make_pair(cp, wl, assoc=assoc)
    z = rng.integers(0, K, size=cp.n_tokens).astype(np.int32)
    r = np.ones(cp.n_tokens, np.uint8)
    z[cp.words == 0] = 0
    if sources:
        s.set_assignments(z, r, np.zeros(cp.n_tokens, np.uint8))
    else:
        s.set_assignments(z, r)
    _, _, B, _ = s.totals()
    assert B[0, 0] == 70000
    for sw in range(2):
        rep, ch, rp = parity.one_step(s, m, sw, 23)
        say(f"  sweep {sw}: {rep}")
    assert s.check() == 0
    s.close()


def test_read_probe_on_a_device_buffer():
    """The read probe measures a device buffer and refuses a range past it."""
    import torch

    from paper_1510_06549_amd import spdp as sp

    say("read probe on a 64 MiB device buffer")
    nbytes = 64 << 20
    buf = torch.ones(nbytes // 4, dtype=torch.int32, device="cuda")
    torch.cuda.synchronize()
    st = torch.cuda.current_stream().cuda_stream
    assert sp.spdp_read_probe(buf.data_ptr(), nbytes, 0, 0, 1024, st) > 0.0
    for rb in (1024, 2048, 3072, 4096, 8192):
        assert sp.spdp_read_probe(buf.data_ptr(), nbytes, rb, nbytes // rb, 512, st) > 0.0
    with pytest.raises(sp.SpdpError) as e:
        sp.spdp_read_probe(buf.data_ptr(), nbytes + 4096, 0, 0, 64, st)
    assert e.value.code == sp.SPDP_E_ARG
    host = np.ones(1 << 16, np.int32)
    with pytest.raises(sp.SpdpError) as e:
        sp.spdp_read_probe(host.ctypes.data, host.nbytes, 0, 0, 64, st)
    assert e.value.code == sp.SPDP_E_ARG
    assert torch.all(buf == 1)


@pytest.mark.parametrize("K", [1, 2, 64, 65, 129, 257, 513, 769, 1024])
def test_narrow_and_wide_rows_at_every_lane_layout(K):
    """Rows of both widths in one corpus: words repeated more than 255 times in
    a group (32-bit rows) beside rare words (16-bit narrow copies), including
    a pair with exactly 255 tokens (the last narrow count) and one with 256,
    at every per-lane topic count of the sampler."""
    say(f"narrow and wide count rows, K = {K}")
    rng = np.random.default_rng(K)
    V = 40
    docs = []
    for d in range(60):
        g = d % 2
        L = int(rng.integers(20, 90))
        # word 0: ~15 per document (wide in both groups); word 1: a tail word
        ws = [0] * 15 + list(rng.integers(2, V, size=L))
        docs.append((g, ws))
    # exactly 255 tokens of word 1 in group 0 and 256 in group 1
    docs.append((0, [1] * 255))
    docs.append((1, [1] * 200))
    docs.append((1, [1] * 56))
    cp = corpus_from_docs(docs, vocab=V)
    q = np.repeat(cp.doc_group, np.diff(cp.doc_off)).astype(np.int64) * V + cp.words
    c = np.bincount(q, minlength=2 * V)
    assert c[1] == 255 and c[V + 1] == 256 and c[0] > 255 and c[V] > 255
    wl = W(K=K)
    s, m = parity.make_pair(cp, wl, init_seed=K)
    for sw in range(3):
        rep, ch, rp = parity.one_step(s, m, sw, 17)
        say(f"  {rep}")
    assert s.check() == 0
    s.close()


def test_stirling_cache_above_23k_customers():
    """A (group, word) pair with 24 000 tokens, above the 23 170 at which the
    fp32 ratio pairs pass 2^31 bytes: the sampler's 32-bit byte offsets into
    them reach 2.3 GB.  Weights, draws and the rebuild match the oracle over
    two sweeps."""
    check_large_pair(24000, 11)


def test_stirling_cache_past_2_29_ratio_pairs():
    """A (group, word) pair with 33 000 tokens: 544 M ratio pairs, past the 2^29
    that 32-bit byte offsets reach, so the samplers' 64-bit-address instance
    runs (17.4 GB of tables).  Weights, draws and the rebuild match the oracle
    over two sweeps; a pair with 65 536 tokens, which 16-bit counts cannot
    hold, is refused with E_RANGE."""
    from paper_1510_06549_amd import spdp as sp

    check_large_pair(33000, 13)
    say("a pair with 65536 tokens is refused")
    words = np.zeros(65536, np.int32)
    with pytest.raises(sp.SpdpError) as e:
        sp.spdp_create(words, np.array([0, 65536], np.int64), np.array([0], np.int32), 1, 2, 3,
                       0.1, 0.5, 1.0, 0.1)
    assert e.value.code == sp.SPDP_E_RANGE


def test_stirling_cache_past_2_29_ratio_pairs_with_word_associations():
    """The association sampler's 64-bit-address instance: the same 33 000-token
    pair under P = 0.7 I + 0.3 Pi (two sources in every row: word 0 lists
    itself and word 4), so new tables of word 0 draw either source.  Weights,
    draws, sources and the rebuild match the oracle over two sweeps."""
    check_large_pair(33000, 18, sources=2)


def check_large_pair(count, seed, sources=0):
    say(f"Stirling cache for {count} customers" + (f", {sources} sources" if sources else ""))
    rng = np.random.default_rng(seed)
    docs = []
    for _ in range(3):
        d = [0] * (count // 3) + list(rng.integers(1, 5, size=30))
        rng.shuffle(d)
        docs.append((0, d))
    cp = corpus_from_docs(docs, vocab=5)
    wl = W(K=3, alpha=0.5, a=0.5, b=20.0, gamma=0.1)
    assoc = synth.associations(1, 5, sources, 0.3, seed) if sources else None
    s, m = parity.make_pair(cp, wl, assoc=assoc)
    assert s.info["ncap"] == count and s.S == sources
    for sw in range(2):
        rep, _, _ = parity.one_step(s, m, sw, 29)
        say(f"  sweep {sw}: {rep}")
    assert s.check() == 0
    s.close()
