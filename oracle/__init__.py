"""fp64 CPU oracle of the SPDP snapshot-parallel Gibbs sweep (ctypes binding).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the CPU
baseline leg of the benchmark, never by the product library.  It shares no code
with the HIP path.  The sampler's arithmetic lives in ``oracle.c``; this module
only marshals numpy arrays.  ``hellinger.py`` (numpy) compares two topic
models.

Model: Li (2012), arXiv:1510.06549, chapter "Shared Topic Modelling Using
Shadow Poisson Dirichlet Process" with identity transformation matrices:
conditionals Eq. SPDP-sampling-w-z-r0 / Eq. SPDP-sampling-w-z-r1, sequential
semantics Algorithm SPDP-Full-Gibbs, joint from the blocked-Gibbs derivation.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
# SPDP_ORACLE_LIB names another build of oracle.c to load instead (the
# sanitizer test runs the pins against an AddressSanitizer/UBSan build)
_LIB_PATH = os.environ.get("SPDP_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")

PURPOSE_SAMPLE = 0
PURPOSE_INIT = 1


def build(force: bool = True) -> str:
    """Compile oracle.c into liboracle.so (gcc, -O2, OpenMP)."""
    if os.environ.get("SPDP_ORACLE_LIB"):
        return _LIB_PATH  # a build made elsewhere (see build_sanitized)
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(
            ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", _SRC, "-lm", "-o", tmp]
        )
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


SANITIZE_FLAGS = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                  "-fno-omit-frame-pointer", "-g", "-O1"]


def build_sanitized(path: str) -> str:
    """Compile oracle.c with AddressSanitizer and UndefinedBehaviorSanitizer
    (host code only) into `path`; load it by setting SPDP_ORACLE_LIB, with
    the ASan runtime preloaded into the interpreter."""
    subprocess.check_call(["gcc", *SANITIZE_FLAGS, "-fopenmp", "-fPIC", "-shared", _SRC, "-lm",
                           "-o", path])
    return path


class _Model(C.Structure):
    _fields_ = [
        ("n_tokens", C.c_int64),
        ("n_docs", C.c_int32),
        ("vocab", C.c_int32),
        ("n_groups", C.c_int32),
        ("K", C.c_int32),
        ("words", C.c_void_p),
        ("doc_off", C.c_void_p),
        ("doc_group", C.c_void_p),
        ("alpha", C.c_double),
        ("a", C.c_double),
        ("b", C.c_double),
        ("gam", C.c_double),
        ("ncap", C.c_int32),
        ("logS", C.c_void_p),
    ]


class _Counts(C.Structure):
    _fields_ = [
        ("n", C.c_void_p),
        ("t", C.c_void_p),
        ("Ngk", C.c_void_p),
        ("Tgk", C.c_void_p),
        ("Bkw", C.c_void_p),
        ("Bk", C.c_void_p),
    ]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=True)
        _lib = _bind(C.CDLL(_LIB_PATH))
    return _lib


class swap_library:
    """Context manager: every call of this module goes to the library at
    `path` (a variant of oracle.c built by a test, e.g. with a planted
    mistake) until the block ends."""

    def __init__(self, path: str):
        self.path = path

    def __enter__(self):
        global _lib
        self._saved = lib()
        _lib = _bind(C.CDLL(self.path))
        return _lib

    def __exit__(self, *exc):
        global _lib
        _lib = self._saved
        return False


def _bind(L):
    """Argument and return types of the library's entry points."""
    vp, i32, i64, u32, u64, dbl = C.c_void_p, C.c_int32, C.c_int64, C.c_uint32, C.c_uint64, C.c_double
    L.or_philox4x32_10.argtypes = [vp, vp, vp]
    L.or_philox4x32_10.restype = None
    L.or_philox_word0.argtypes = [u64, i64, u32, u32]
    L.or_philox_word0.restype = u32
    L.or_uniform.argtypes = [u64, i64, u32]
    L.or_uniform.restype = dbl
    L.or_stirling_log_table.argtypes = [i32, dbl, vp]
    L.or_stirling_log_table.restype = C.c_int
    L.or_init.argtypes = [vp, u64, vp, vp]
    L.or_init.restype = None
    L.or_rebuild.argtypes = [vp, vp, vp, vp]
    L.or_rebuild.restype = None
    L.or_repair.argtypes = [vp, vp, vp, vp]
    L.or_repair.restype = i64
    L.or_token_weights.argtypes = [vp, vp, vp, i32, i32, i32, i32, vp]
    L.or_token_weights.restype = C.c_int
    L.or_sample_docs.argtypes = [vp, vp, vp, vp, u32, u64, i32, i32, vp, vp, vp, i64, i64]
    L.or_sample_docs.restype = i64
    L.or_sweep.argtypes = [vp, vp, vp, vp, u32, u64, C.c_int, vp]
    L.or_sweep.restype = C.c_int
    L.or_loglik.argtypes = [vp, vp, vp, vp]
    L.or_loglik.restype = dbl
    L.or_max_group_word_count.argtypes = [vp]
    L.or_max_group_word_count.restype = i32
    L.or_chain_histogram.argtypes = [vp, vp, vp, vp, u32, i64, u64, C.c_int, vp, i64]
    L.or_chain_histogram.restype = C.c_int
    L.or_interleaved_order.argtypes = [vp, vp]
    L.or_interleaved_order.restype = None
    L.or_sweep_ordered.argtypes = [vp, vp, vp, vp, u32, u64, vp, C.c_int, vp]
    L.or_sweep_ordered.restype = C.c_int
    L.or_chain_histogram_ordered.argtypes = [vp, vp, vp, vp, u32, i64, u64, vp, vp, i64]
    L.or_chain_histogram_ordered.restype = C.c_int
    L.or_num_threads.argtypes = []
    L.or_num_threads.restype = C.c_int
    L.or_set_num_threads.argtypes = [C.c_int]
    L.or_set_num_threads.restype = C.c_int
    L.or_estimates.argtypes = [vp, vp, vp, vp, vp, vp]
    L.or_estimates.restype = None
    L.or_heldout.argtypes = [vp, vp, i32, vp, vp, vp, i32, u64, vp, vp]
    L.or_heldout.restype = dbl
    L.or_head_source.argtypes = [vp, vp, i32, i32]
    L.or_head_source.restype = i32
    L.or_rebuild_assoc.argtypes = [vp, vp, vp, vp, vp, vp]
    L.or_rebuild_assoc.restype = None
    L.or_repair_assoc.argtypes = [vp, vp, vp, vp, vp, vp]
    L.or_repair_assoc.restype = i64
    L.or_token_weights_assoc.argtypes = [vp, vp, vp, vp, i32, i32, i32, i32, i32, vp]
    L.or_token_weights_assoc.restype = C.c_int
    L.or_sample_docs_assoc.argtypes = [vp, vp, vp, vp, vp, vp, u32, u64, i32, i32, vp, vp,
                                       vp, i64, i64]
    L.or_sample_docs_assoc.restype = i64
    L.or_sweep_assoc.argtypes = [vp, vp, vp, vp, vp, vp, u32, u64, C.c_int, vp]
    L.or_sweep_assoc.restype = C.c_int
    L.or_loglik_assoc.argtypes = [vp, vp, vp, vp, vp, vp]
    L.or_loglik_assoc.restype = dbl
    L.or_estimates_assoc.argtypes = [vp, vp, vp, vp, vp, vp, vp]
    L.or_estimates_assoc.restype = None
    L.or_chain_histogram_assoc.argtypes = [vp, vp, vp, vp, vp, vp, u32, i64, u64, C.c_int,
                                           vp, i64]
    L.or_chain_histogram_assoc.restype = C.c_int
    return L


def _p(a: np.ndarray):
    return a.ctypes.data_as(C.c_void_p)


# --------------------------------------------------------------------------
# Philox and Stirling
# --------------------------------------------------------------------------
def philox4x32_10(ctr, key) -> np.ndarray:
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    lib().or_philox4x32_10(_p(c), _p(k), _p(out))
    return out


def philox_word0(seed: int, i: int, sweep: int, purpose: int) -> int:
    return int(lib().or_philox_word0(seed, i, sweep, purpose))


def uniform(seed: int, i: int, sweep: int) -> float:
    return float(lib().or_uniform(seed, i, sweep))


def stirling_log_table(nmax: int, a: float) -> np.ndarray:
    """Triangle of log S^n_{t,a}, 0 <= t <= n <= nmax; row n starts at n(n+1)/2."""
    out = np.empty((nmax + 1) * (nmax + 2) // 2, dtype=np.float64)
    if lib().or_stirling_log_table(nmax, a, _p(out)) != 0:
        raise ValueError("bad Stirling table arguments")
    return out


def tri(n: int, t: int) -> int:
    return n * (n + 1) // 2 + t


# --------------------------------------------------------------------------
# Model + counts
# --------------------------------------------------------------------------
class Model:
    """A corpus with hyperparameters and the fp64 Stirling table it needs."""

    def __init__(self, words, doc_off, doc_group, n_groups, K, vocab, alpha, a, b, gamma,
                 ncap: int | None = None):
        self.words = np.ascontiguousarray(words, dtype=np.int32)
        self.doc_off = np.ascontiguousarray(doc_off, dtype=np.int64)
        self.doc_group = np.ascontiguousarray(doc_group, dtype=np.int32)
        self.N = int(self.words.shape[0])
        self.D = int(self.doc_group.shape[0])
        self.G, self.K, self.V = int(n_groups), int(K), int(vocab)
        self.alpha, self.a, self.b, self.gamma = float(alpha), float(a), float(b), float(gamma)
        assert self.doc_off.shape[0] == self.D + 1 and self.doc_off[-1] == self.N
        self._m = _Model()
        m = self._m
        m.n_tokens, m.n_docs, m.vocab, m.n_groups, m.K = self.N, self.D, self.V, self.G, self.K
        m.words, m.doc_off, m.doc_group = (_p(self.words).value, _p(self.doc_off).value,
                                           _p(self.doc_group).value)
        m.alpha, m.a, m.b, m.gam = self.alpha, self.a, self.b, self.gamma
        if ncap is None:
            ncap = int(lib().or_max_group_word_count(C.byref(m))) if self.N else 0
        self.ncap = int(ncap)
        self.logS = stirling_log_table(self.ncap + 1, self.a)
        m.ncap = self.ncap + 1
        m.logS = _p(self.logS).value

    @property
    def ref(self):
        return C.byref(self._m)

    def new_counts(self) -> "Counts":
        return Counts(self.G, self.K, self.V)

    # ---- operations ----
    def init(self, init_seed: int):
        z = np.empty(self.N, dtype=np.int32)
        r = np.empty(self.N, dtype=np.uint8)
        lib().or_init(self.ref, init_seed, _p(z), _p(r))
        return z, r

    def rebuild(self, z, r, counts: "Counts | None" = None) -> "Counts":
        c = counts if counts is not None else self.new_counts()
        lib().or_rebuild(self.ref, _p(z), _p(r), c.ref)
        return c

    def repair(self, z, r, counts: "Counts") -> int:
        return int(lib().or_repair(self.ref, _p(z), _p(r), counts.ref))

    def initial_state(self, init_seed: int):
        """Philox-uniform topics, r = 0, rebuild, repair (one head per non-empty cell)."""
        z, r = self.init(init_seed)
        c = self.rebuild(z, r)
        self.repair(z, r, c)
        return z, r, c

    def token_weights(self, counts: "Counts", crow, g, w, k0, r0):
        """2K weights (None if the sole-head point mass applies)."""
        out = np.zeros(2 * self.K, dtype=np.float64)
        crow = np.ascontiguousarray(crow, dtype=np.int32)
        skip = lib().or_token_weights(self.ref, counts.ref, _p(crow), int(g), int(w), int(k0),
                                      int(r0), _p(out))
        return None if skip else out

    def sample_docs(self, counts, z, r, sweep, seed, d_begin=0, d_end=None, trace=None):
        """Sampling step over documents [d_begin, d_end) against `counts` (read only).

        trace = (tok_begin, tok_end) returns (changed, w[T,2K], u[T], skip[T]).
        """
        if d_end is None:
            d_end = self.D
        if trace is None:
            ch = lib().or_sample_docs(self.ref, counts.ref, _p(z), _p(r), sweep, seed, d_begin,
                                      d_end, None, None, None, 0, 0)
            return int(ch)
        tb, te = trace
        T = te - tb
        tw = np.zeros((T, 2 * self.K), dtype=np.float64)
        tu = np.full(T, np.nan, dtype=np.float64)
        ts = np.zeros(T, dtype=np.uint8)
        ch = lib().or_sample_docs(self.ref, counts.ref, _p(z), _p(r), sweep, seed, d_begin, d_end,
                                  _p(tw), _p(tu), _p(ts), tb, te)
        return int(ch), tw, tu, ts

    def interleaved_order(self):
        """Visiting order of the word order rearrangement: round robin over the
        position inside the document, documents in index order."""
        order = np.zeros(self.N, dtype=np.int32)
        lib().or_interleaved_order(self.ref, _p(order))
        return order

    def sweep(self, counts, z, r, sweep, seed, mode: str = "snapshot", order=None,
              stale_totals=False):
        """mode "snapshot", "sequential" (token index order) or "ordered"
        (sequential in the visiting order `order`; stale_totals holds the sums
        N_gk, T_gk, B_k at their sweep-start values in the conditionals)."""
        stats = np.zeros(2, dtype=np.int64)
        if mode == "ordered":
            order = np.ascontiguousarray(order, dtype=np.int32)
            assert order.shape == (self.N,)
            rc = lib().or_sweep_ordered(self.ref, counts.ref, _p(z), _p(r), sweep, seed,
                                        _p(order), 1 if stale_totals else 0, _p(stats))
        else:
            rc = lib().or_sweep(self.ref, counts.ref, _p(z), _p(r), sweep, seed,
                                0 if mode == "snapshot" else 1, _p(stats))
        if rc != 0:
            raise ValueError(mode)
        return int(stats[0]), int(stats[1])

    def chain_histogram(self, counts, z, r, first_sweep, n_sweeps, seed, mode="sequential",
                        order=None):
        """Visit counts of encoded states over `n_sweeps` sweeps (tiny corpora only)."""
        n_bins = (2 * self.K) ** self.N
        hist = np.zeros(n_bins, dtype=np.int64)
        if mode == "ordered":
            order = np.ascontiguousarray(order, dtype=np.int32)
            rc = lib().or_chain_histogram_ordered(self.ref, counts.ref, _p(z), _p(r),
                                                  first_sweep, n_sweeps, seed, _p(order),
                                                  _p(hist), n_bins)
        else:
            rc = lib().or_chain_histogram(self.ref, counts.ref, _p(z), _p(r), first_sweep,
                                          n_sweeps, seed, 0 if mode == "snapshot" else 1,
                                          _p(hist), n_bins)
        if rc != 0:
            raise RuntimeError(f"or_chain_histogram failed ({rc})")
        return hist

    def loglik(self, z, r, counts: "Counts") -> float:
        return float(lib().or_loglik(self.ref, _p(z), _p(r), counts.ref))

    def estimates(self, z, counts: "Counts"):
        """Point estimates (theta [D, K], phi0 [K, V], phig [G, K, V]) of a state."""
        theta = np.zeros((self.D, self.K), dtype=np.float64)
        phi0 = np.zeros((self.K, self.V), dtype=np.float64)
        phig = np.zeros((self.G, self.K, self.V), dtype=np.float64)
        lib().or_estimates(self.ref, _p(np.ascontiguousarray(z, dtype=np.int32)), counts.ref,
                           _p(theta), _p(phi0), _p(phig))
        return theta, phi0, phig

    def heldout(self, phig, words, doc_off, doc_group, n_sweeps: int, seed: int):
        """Fold-in of held-out documents with phi fixed at `phig` [G, K, V].

        Returns (sum of log p(w_d), final topics z [N_test], log p per document).
        """
        phig = np.ascontiguousarray(phig, dtype=np.float64)
        assert phig.shape == (self.G, self.K, self.V)
        words = np.ascontiguousarray(words, dtype=np.int32)
        doc_off = np.ascontiguousarray(doc_off, dtype=np.int64)
        doc_group = np.ascontiguousarray(doc_group, dtype=np.int32)
        D = int(doc_group.shape[0])
        assert doc_off.shape[0] == D + 1 and doc_off[-1] == words.shape[0]
        assert words.size == 0 or (words.min() >= 0 and words.max() < self.V)
        assert D == 0 or (doc_group.min() >= 0 and doc_group.max() < self.G)
        z = np.zeros(words.shape[0], dtype=np.int32)
        ll_doc = np.zeros(D, dtype=np.float64)
        total = lib().or_heldout(self.ref, _p(phig), D, _p(words), _p(doc_off), _p(doc_group),
                                 int(n_sweeps), int(seed) & (2**64 - 1), _p(z), _p(ll_doc))
        return float(total), z, ll_doc


class _Assoc(C.Structure):
    _fields_ = [
        ("S", C.c_int32),
        ("row_off", C.c_void_p),
        ("src", C.c_void_p),
        ("p", C.c_void_p),
    ]


class AssocModel(Model):
    """The model with word associations (non-identity P^g): every head carries
    the slot s of its source in its row's list, and the shadow-base counts
    Bkw[k, v] are keyed by source.  `row_off` [G V + 1] int64, `src` [nnz]
    int32 and `p` [nnz] float64 list, for each row (g, w) in order, the
    sources v with p_{g,w,v} > 0."""

    def __init__(self, words, doc_off, doc_group, n_groups, K, vocab, alpha, a, b, gamma,
                 row_off, src, p, ncap: int | None = None):
        super().__init__(words, doc_off, doc_group, n_groups, K, vocab, alpha, a, b, gamma, ncap)
        self.row_off = np.ascontiguousarray(row_off, dtype=np.int64)
        self.src = np.ascontiguousarray(src, dtype=np.int32)
        self.p = np.ascontiguousarray(p, dtype=np.float64)
        assert self.row_off.shape == (self.G * self.V + 1,) and self.row_off[0] == 0
        assert self.row_off[-1] == self.src.shape[0] == self.p.shape[0]
        lens = np.diff(self.row_off)
        assert lens.min() >= 1, "every row needs a source"
        self.S = int(lens.max())
        self._a = _Assoc(self.S, _p(self.row_off).value, _p(self.src).value, _p(self.p).value)

    @property
    def aref(self):
        return C.byref(self._a)

    def head_source(self, g, w) -> int:
        return int(lib().or_head_source(self.ref, self.aref, int(g), int(w)))

    def rebuild(self, z, r, s, counts: "Counts | None" = None) -> "Counts":
        c = counts if counts is not None else self.new_counts()
        lib().or_rebuild_assoc(self.ref, self.aref, _p(z), _p(r), _p(s), c.ref)
        return c

    def repair(self, z, r, s, counts: "Counts") -> int:
        return int(lib().or_repair_assoc(self.ref, self.aref, _p(z), _p(r), _p(s), counts.ref))

    def initial_state(self, init_seed: int):
        """Philox-uniform topics, r = 0, s = 0, rebuild, repair."""
        z, r = self.init(init_seed)
        s = np.zeros(self.N, dtype=np.uint8)
        c = self.rebuild(z, r, s)
        self.repair(z, r, s, c)
        return z, r, s, c

    def token_weights(self, counts, crow, g, w, k0, r0, s0):
        """K (S + 1) weights (None if the sole-head point mass applies)."""
        out = np.zeros(self.K * (self.S + 1), dtype=np.float64)
        crow = np.ascontiguousarray(crow, dtype=np.int32)
        skip = lib().or_token_weights_assoc(self.ref, self.aref, counts.ref, _p(crow), int(g),
                                            int(w), int(k0), int(r0), int(s0), _p(out))
        return None if skip else out

    def sample_docs(self, counts, z, r, s, sweep, seed, d_begin=0, d_end=None, trace=None):
        if d_end is None:
            d_end = self.D
        if trace is None:
            return int(lib().or_sample_docs_assoc(self.ref, self.aref, counts.ref, _p(z), _p(r),
                                                  _p(s), sweep, seed, d_begin, d_end, None, None,
                                                  None, 0, 0))
        tb, te = trace
        T = te - tb
        tw = np.zeros((T, self.K * (self.S + 1)), dtype=np.float64)
        tu = np.full(T, np.nan, dtype=np.float64)
        ts = np.zeros(T, dtype=np.uint8)
        ch = lib().or_sample_docs_assoc(self.ref, self.aref, counts.ref, _p(z), _p(r), _p(s),
                                        sweep, seed, d_begin, d_end, _p(tw), _p(tu), _p(ts), tb,
                                        te)
        return int(ch), tw, tu, ts

    def sweep(self, counts, z, r, s, sweep, seed, mode: str = "snapshot"):
        stats = np.zeros(2, dtype=np.int64)
        rc = lib().or_sweep_assoc(self.ref, self.aref, counts.ref, _p(z), _p(r), _p(s), sweep,
                                  seed, 0 if mode == "snapshot" else 1, _p(stats))
        if rc != 0:
            raise ValueError(mode)
        return int(stats[0]), int(stats[1])

    def chain_histogram(self, counts, z, r, s, first_sweep, n_sweeps, seed, mode="sequential"):
        n_bins = (self.K * (self.S + 1)) ** self.N
        hist = np.zeros(n_bins, dtype=np.int64)
        rc = lib().or_chain_histogram_assoc(self.ref, self.aref, counts.ref, _p(z), _p(r), _p(s),
                                            first_sweep, n_sweeps, seed,
                                            0 if mode == "snapshot" else 1, _p(hist), n_bins)
        if rc != 0:
            raise RuntimeError(f"or_chain_histogram_assoc failed ({rc})")
        return hist

    def loglik(self, z, r, s, counts: "Counts") -> float:
        return float(lib().or_loglik_assoc(self.ref, self.aref, _p(z), _p(r), _p(s), counts.ref))

    def estimates(self, z, counts: "Counts"):
        theta = np.zeros((self.D, self.K), dtype=np.float64)
        phi0 = np.zeros((self.K, self.V), dtype=np.float64)
        phig = np.zeros((self.G, self.K, self.V), dtype=np.float64)
        lib().or_estimates_assoc(self.ref, self.aref,
                                 _p(np.ascontiguousarray(z, dtype=np.int32)), counts.ref,
                                 _p(theta), _p(phi0), _p(phig))
        return theta, phi0, phig


class Counts:
    """Count arrays in the thesis's logical layout: n[g, k, w], t[g, k, w]."""

    def __init__(self, G, K, V):
        self.n = np.zeros((G, K, V), dtype=np.int32)
        self.t = np.zeros((G, K, V), dtype=np.int32)
        self.Ngk = np.zeros((G, K), dtype=np.int32)
        self.Tgk = np.zeros((G, K), dtype=np.int32)
        self.Bkw = np.zeros((K, V), dtype=np.int32)
        self.Bk = np.zeros(K, dtype=np.int32)
        self._c = _Counts(_p(self.n).value, _p(self.t).value, _p(self.Ngk).value,
                          _p(self.Tgk).value, _p(self.Bkw).value, _p(self.Bk).value)

    @property
    def ref(self):
        return C.byref(self._c)

    def copy(self) -> "Counts":
        c = Counts(*self.n.shape)
        for f in ("n", "t", "Ngk", "Tgk", "Bkw", "Bk"):
            getattr(c, f)[...] = getattr(self, f)
        return c


def num_threads() -> int:
    return int(lib().or_num_threads())


def set_num_threads(n: int) -> int:
    """Threads of the oracle's OpenMP loops from now on; returns the new count."""
    return int(lib().or_set_num_threads(int(n)))


from .hellinger import align_topics, hellinger  # noqa: E402  (topic-model comparison)
