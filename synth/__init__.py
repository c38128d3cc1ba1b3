"""Seeded synthetic SPDP corpora (input generator for tests and the benchmark).

Draws corpora from the SPDP generative process (see ``synth.c``).  This module
holds no sampler arithmetic; it only builds and calls the C generator and
describes the five workloads the sweep is exercised on.  The thesis's own
corpora (RedState/DailyKos blogs, Reuters RCV1 subsets) are not available, so
these synthetic corpora of matching structure stand in for them.
"""
from __future__ import annotations

import ctypes as C
import dataclasses
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "synth.c")
_LIB_PATH = os.path.join(_HERE, "libsynth.so")


def build(force: bool = True) -> str:
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(
            ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", _SRC, "-lm", "-o", tmp]
        )
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


class _Params(C.Structure):
    _fields_ = [
        ("n_groups", C.c_int32),
        ("docs_per_group", C.c_int32),
        ("vocab", C.c_int32),
        ("K", C.c_int32),
        ("doc_len_mean", C.c_double),
        ("zipf_s", C.c_double),
        ("alpha", C.c_double),
        ("a", C.c_double),
        ("b", C.c_double),
    ]


_lib = None


def _L():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=True)
        L = C.CDLL(_LIB_PATH)
        L.synth_doc_lengths.argtypes = [C.c_void_p, C.c_uint64, C.c_void_p]
        L.synth_doc_lengths.restype = C.c_int64
        L.synth_fill.argtypes = [C.c_void_p, C.c_uint64, C.c_void_p, C.c_void_p, C.c_void_p,
                                 C.c_void_p]
        L.synth_fill.restype = C.c_int
        L.synth_phi0.argtypes = [C.c_void_p, C.c_uint64, C.c_void_p]
        L.synth_phi0.restype = C.c_int
        _lib = L
    return _lib


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic workload: corpus shape plus inference hyperparameters."""

    name: str
    n_groups: int
    docs_per_group: int
    doc_len_mean: float
    vocab: int
    zipf_s: float
    K: int
    alpha: float
    a: float
    b: float
    gamma: float
    sweeps: int

    def scaled(self, docs_per_group: int) -> "Workload":
        return dataclasses.replace(self, name=f"{self.name}-d{docs_per_group}",
                                   docs_per_group=docs_per_group)


# The five workloads: shapes of the thesis's corpora (2-4 groups, 1k-7k docs a
# group, 100-250 tokens a doc, 15k-156k words) scaled from a tiny parity case
# up to one that fills HBM with 8 GB of dense counts.
WORKLOADS = [
    Workload("g2-d100-k10", 2, 100, 50.0, 1000, 1.1, 10, 0.1, 0.5, 10.0, 0.01, 50),
    Workload("g2-d1000-k50", 2, 1000, 100.0, 5000, 1.1, 50, 0.1, 0.5, 10.0, 0.01, 200),
    Workload("g4-d5000-k100", 4, 5000, 150.0, 20000, 1.05, 100, 0.05, 0.7, 50.0, 0.01, 100),
    Workload("g10-d20000-k200", 10, 20000, 200.0, 50000, 1.05, 200, 0.05, 0.7, 50.0, 0.005, 20),
    Workload("g20-d50000-k500", 20, 50000, 250.0, 100000, 1.0, 500, 0.02, 0.8, 100.0, 0.005, 10),
]


def workload(idx_or_name) -> Workload:
    if isinstance(idx_or_name, int):
        return WORKLOADS[idx_or_name]
    for w in WORKLOADS:
        if w.name == idx_or_name:
            return w
    raise KeyError(idx_or_name)


@dataclasses.dataclass
class Corpus:
    words: np.ndarray      # int32 [N]
    doc_off: np.ndarray    # int64 [D+1]
    doc_group: np.ndarray  # int32 [D]
    z_true: np.ndarray     # int32 [N] generating topics
    r_true: np.ndarray     # uint8 [N] generating table indicators
    n_groups: int
    vocab: int

    @property
    def n_tokens(self) -> int:
        return int(self.words.shape[0])

    @property
    def n_docs(self) -> int:
        return int(self.doc_group.shape[0])


def generate(w: Workload, seed: int = 0) -> Corpus:
    """Draw a corpus for workload `w` (deterministic in `seed`, any thread count)."""
    p = _Params(w.n_groups, w.docs_per_group, w.vocab, w.K, w.doc_len_mean, w.zipf_s,
                w.alpha, w.a, w.b)
    D = w.n_groups * w.docs_per_group
    lens = np.empty(D, dtype=np.int32)
    N = int(_L().synth_doc_lengths(C.byref(p), seed, lens.ctypes.data))
    doc_off = np.zeros(D + 1, dtype=np.int64)
    np.cumsum(lens, out=doc_off[1:])
    assert doc_off[-1] == N
    words = np.empty(N, dtype=np.int32)
    z = np.empty(N, dtype=np.int32)
    r = np.empty(N, dtype=np.uint8)
    rc = _L().synth_fill(C.byref(p), seed, doc_off.ctypes.data, words.ctypes.data,
                         z.ctypes.data, r.ctypes.data)
    if rc != 0:
        raise MemoryError("synth_fill failed")
    doc_group = (np.arange(D, dtype=np.int64) // w.docs_per_group).astype(np.int32)
    return Corpus(words, doc_off, doc_group, z, r, w.n_groups, w.vocab)


def true_phi0(w: Workload, seed: int = 0) -> np.ndarray:
    """The generating shadow base phi0 [K, V] of ``generate(w, seed)``: the law
    from which a new table of topic k draws its word."""
    p = _Params(w.n_groups, w.docs_per_group, w.vocab, w.K, w.doc_len_mean, w.zipf_s,
                w.alpha, w.a, w.b)
    out = np.empty((w.K, w.vocab), dtype=np.float64)
    if _L().synth_phi0(C.byref(p), seed, out.ctypes.data) != 0:
        raise MemoryError("synth_phi0 failed")
    return out


def associations(n_groups: int, vocab: int, S: int, eps: float, seed: int = 0):
    """Sparse word-association matrices P^g, one per group (the transformation
    matrices of the model with word associations): P^g = (1 - eps) I +
    eps / (S - 1) sum_{j < S-1} Pi_{g,j}, with Pi a seeded random permutation
    matrix (Pi[w][v] = 1 iff w = pi(v)), so every row and every column sums to
    one and row w lists at most S sources: w itself, then pi_j^{-1}(w) for
    j = 0, 1, ... (a repeated source is merged into its first entry).  S = 1
    gives the identity.  Returns CSR arrays over the rows (g, w) in order:
    (row_off [G V + 1] int64, src [nnz] int32, p [nnz] float64)."""
    if S < 1 or not 0.0 <= eps < 1.0:
        raise ValueError("need S >= 1 and 0 <= eps < 1")
    rng = np.random.default_rng([seed, 0xA550C])
    rows_src, rows_p, lens = [], [], []
    w = np.arange(vocab)
    for _ in range(n_groups):
        cand = np.empty((vocab, S), dtype=np.int64)
        val = np.empty((vocab, S), dtype=np.float64)
        cand[:, 0], val[:, 0] = w, (1.0 - eps) if S > 1 else 1.0
        for j in range(1, S):
            perm = rng.permutation(vocab)
            inv = np.empty(vocab, dtype=np.int64)
            inv[perm] = w
            cand[:, j], val[:, j] = inv, eps / (S - 1)
        keep = np.ones((vocab, S), dtype=bool)
        for j in range(1, S):
            for i in range(j):
                same = keep[:, j] & (cand[:, j] == cand[:, i]) & keep[:, i]
                val[same, i] += val[same, j]
                keep[same, j] = False
        lens.append(keep.sum(1))
        rows_src.append(cand[keep])
        rows_p.append(val[keep])
    lens = np.concatenate(lens) if n_groups else np.zeros(0, dtype=np.int64)
    row_off = np.zeros(n_groups * vocab + 1, dtype=np.int64)
    np.cumsum(lens, out=row_off[1:])
    src = np.concatenate(rows_src).astype(np.int32) if n_groups else np.zeros(0, np.int32)
    p = np.concatenate(rows_p) if n_groups else np.zeros(0, np.float64)
    return row_off, src, p


def split_heldout(cp: Corpus, frac: float = 0.1):
    """(train, test): the last floor(frac * docs) documents of every group held out,
    as the thesis holds out 10% of each group for perplexity; both keep corpus
    order, and the test corpus numbers its tokens from 0."""
    test_mask = np.zeros(cp.n_docs, dtype=bool)
    for g in range(cp.n_groups):
        docs = np.flatnonzero(cp.doc_group == g)
        n_out = int(np.floor(frac * docs.size))
        if n_out:
            test_mask[docs[-n_out:]] = True

    def take(mask):
        idx = np.flatnonzero(mask)
        lens = (cp.doc_off[1:] - cp.doc_off[:-1])[idx]
        off = np.zeros(idx.size + 1, dtype=np.int64)
        np.cumsum(lens, out=off[1:])
        tok = np.concatenate([np.arange(cp.doc_off[d], cp.doc_off[d + 1]) for d in idx]) \
            if idx.size else np.zeros(0, dtype=np.int64)
        return Corpus(cp.words[tok].astype(np.int32), off, cp.doc_group[idx].astype(np.int32),
                      cp.z_true[tok].astype(np.int32), cp.r_true[tok].astype(np.uint8),
                      cp.n_groups, cp.vocab)

    return take(~test_mask), take(test_mask)
