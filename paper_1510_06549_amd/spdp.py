"""ctypes binding of libspdp.so (the C ABI declared in include/spdp.h).

Argument marshalling only: every step of the sweep runs in the library's HIP
kernels.  Host buffers are numpy arrays (``where = 0``); device buffers are
torch tensors on the GPU (``where = 1``).  The library is required: importing
this module raises if ``libspdp.so`` has not been built.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libspdp.so")

SPDP_OK = 0
SPDP_E_ARG = -1
SPDP_E_NOMEM = -2
SPDP_E_HIP = -3
SPDP_E_RANGE = -4
SPDP_E_STATE = -5
SPDP_MAX_K = 1024
SPDP_MAX_SOURCES = 8
SPDP_NKERNELS = 4
KERNEL_CLASSES = ("sample", "rebuild", "base", "totals")

# Every entry point of include/spdp.h, in declaration order.
EXPORTS = (
    "spdp_create", "spdp_sweep", "spdp_counts", "spdp_totals", "spdp_loglik", "spdp_destroy",
    "spdp_get_assignments", "spdp_set_assignments", "spdp_debug_conditionals", "spdp_stats",
    "spdp_kernel_timing", "spdp_kernel_times", "spdp_info", "spdp_last_error",
    "spdp_estimates", "spdp_heldout", "spdp_hellinger", "spdp_align_topics",
    "spdp_create_assoc", "spdp_get_slots", "spdp_set_assignments_assoc", "spdp_max_sources",
    "spdp_sweep_async", "spdp_read_probe", "spdp_check", "spdp_debug_poke",
    "spdp_hellinger_noalloc",
)


class SpdpError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"spdp error {code}: {msg}")
        self.code = code


class _Corpus(C.Structure):
    _fields_ = [
        ("n_tokens", C.c_int64),
        ("n_docs", C.c_int32),
        ("vocab", C.c_int32),
        ("words", C.c_void_p),
        ("doc_offsets", C.c_void_p),
        ("init_seed", C.c_uint64),
        ("hip_stream", C.c_void_p),
    ]


class _Groups(C.Structure):
    _fields_ = [("n_groups", C.c_int32), ("doc_group", C.c_void_p)]


class _Assoc(C.Structure):
    _fields_ = [
        ("max_sources", C.c_int32),
        ("row_off", C.c_void_p),
        ("src", C.c_void_p),
        ("p", C.c_void_p),
    ]


def load_library() -> C.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it with `python -c 'import __graft_entry__ as g; "
            f"g.build()'` (hipcc, gfx950) -- there is no fallback implementation")
    L = C.CDLL(LIB_PATH)
    vp, i32, i64, u32, u64, dbl = C.c_void_p, C.c_int32, C.c_int64, C.c_uint32, C.c_uint64, C.c_double
    cint = C.c_int
    L.spdp_create.argtypes = [vp, vp, i32, dbl, dbl, dbl, dbl, C.POINTER(vp)]
    L.spdp_create.restype = cint
    L.spdp_sweep.argtypes = [vp, u32, u64]
    L.spdp_sweep.restype = cint
    L.spdp_counts.argtypes = [vp, i32, i32, vp, vp, cint]
    L.spdp_counts.restype = cint
    L.spdp_totals.argtypes = [vp, vp, vp, vp, vp, cint]
    L.spdp_totals.restype = cint
    L.spdp_loglik.argtypes = [vp, C.POINTER(dbl)]
    L.spdp_loglik.restype = cint
    L.spdp_destroy.argtypes = [vp]
    L.spdp_destroy.restype = None
    L.spdp_get_assignments.argtypes = [vp, vp, vp, cint]
    L.spdp_get_assignments.restype = cint
    L.spdp_set_assignments.argtypes = [vp, vp, vp, cint]
    L.spdp_set_assignments.restype = cint
    L.spdp_debug_conditionals.argtypes = [vp, u32, u64, i64, i64, vp, vp, vp, cint]
    L.spdp_debug_conditionals.restype = cint
    L.spdp_stats.argtypes = [vp, C.POINTER(i64), C.POINTER(i64)]
    L.spdp_stats.restype = cint
    L.spdp_kernel_timing.argtypes = [vp, cint]
    L.spdp_kernel_timing.restype = cint
    L.spdp_kernel_times.argtypes = [vp, vp, vp]
    L.spdp_kernel_times.restype = cint
    L.spdp_info.argtypes = [vp, vp]
    L.spdp_info.restype = cint
    L.spdp_read_probe.argtypes = [vp, i64, cint, i64, cint, vp, vp]
    L.spdp_read_probe.restype = cint
    L.spdp_last_error.argtypes = []
    L.spdp_last_error.restype = C.c_char_p
    L.spdp_estimates.argtypes = [vp, i32, i32, vp, vp, vp, cint]
    L.spdp_estimates.restype = cint
    L.spdp_heldout.argtypes = [vp, vp, vp, i32, u64, vp, vp, cint]
    L.spdp_heldout.restype = cint
    L.spdp_hellinger.argtypes = [vp, vp, i32, vp, i32, i32, vp, cint]
    L.spdp_hellinger.restype = cint
    L.spdp_align_topics.argtypes = [vp, i32, i32, vp, vp]
    L.spdp_align_topics.restype = cint
    L.spdp_create_assoc.argtypes = [vp, vp, vp, i32, dbl, dbl, dbl, dbl, C.POINTER(vp)]
    L.spdp_create_assoc.restype = cint
    L.spdp_get_slots.argtypes = [vp, vp, cint]
    L.spdp_get_slots.restype = cint
    L.spdp_set_assignments_assoc.argtypes = [vp, vp, vp, vp, cint]
    L.spdp_set_assignments_assoc.restype = cint
    L.spdp_max_sources.argtypes = [vp, C.POINTER(i32)]
    L.spdp_max_sources.restype = cint
    L.spdp_sweep_async.argtypes = [vp, u32, u64, i32, i32]
    L.spdp_sweep_async.restype = cint
    L.spdp_hellinger_noalloc.argtypes = [vp, vp, i32, vp, i32, i32, vp]
    L.spdp_hellinger_noalloc.restype = cint
    L.spdp_check.argtypes = [vp, C.POINTER(i64)]
    L.spdp_check.restype = cint
    L.spdp_debug_poke.argtypes = [vp, i32, i32, i32, i32, i32]
    L.spdp_debug_poke.restype = cint
    return L


_lib = None


def lib() -> C.CDLL:
    global _lib
    if _lib is None:
        _lib = load_library()
    return _lib


def spdp_last_error() -> str:
    return lib().spdp_last_error().decode()


def _check(rc: int):
    if rc != SPDP_OK:
        raise SpdpError(rc, spdp_last_error())


def _buf(x):
    """(pointer, where) of a numpy array (host) or a torch CUDA tensor (device)."""
    if x is None:
        return None, 0
    if isinstance(x, np.ndarray):
        assert x.flags.c_contiguous
        return x.ctypes.data, 0
    # torch tensor
    assert x.is_contiguous()
    return x.data_ptr(), (1 if x.is_cuda else 0)


def _where(*bufs) -> int:
    ws = {w for p, w in (_buf(b) for b in bufs) if p is not None}
    if len(ws) > 1:
        raise ValueError("mix of host and device buffers in one call")
    return ws.pop() if ws else 0


# ---------------------------------------------------------------------------
# Entry points (same names as the C ABI)
# ---------------------------------------------------------------------------
def spdp_create(words, doc_offsets, doc_group, n_groups, vocab, K, alpha, a, b, gamma,
                init_seed=0, hip_stream=None):
    words = np.ascontiguousarray(words, dtype=np.int32)
    doc_offsets = np.ascontiguousarray(doc_offsets, dtype=np.int64)
    doc_group = np.ascontiguousarray(doc_group, dtype=np.int32)
    corpus = _Corpus(int(words.shape[0]), int(doc_group.shape[0]), int(vocab), words.ctypes.data,
                     doc_offsets.ctypes.data, int(init_seed) & (2**64 - 1),
                     None if hip_stream is None else int(hip_stream))
    groups = _Groups(int(n_groups), doc_group.ctypes.data)
    h = C.c_void_p()
    _check(lib().spdp_create(C.byref(corpus), C.byref(groups), int(K), float(alpha), float(a),
                             float(b), float(gamma), C.byref(h)))
    return h


def spdp_create_assoc(words, doc_offsets, doc_group, n_groups, vocab, K, alpha, a, b, gamma,
                      row_off, src, p, max_sources=None, init_seed=0, hip_stream=None):
    """State of the model with word associations: row q = g V + w of P^g lists
    its sources src[row_off[q]:row_off[q+1]] with probabilities p (see
    include/spdp.h)."""
    words = np.ascontiguousarray(words, dtype=np.int32)
    doc_offsets = np.ascontiguousarray(doc_offsets, dtype=np.int64)
    doc_group = np.ascontiguousarray(doc_group, dtype=np.int32)
    row_off = np.ascontiguousarray(row_off, dtype=np.int64)
    src = np.ascontiguousarray(src, dtype=np.int32)
    p = np.ascontiguousarray(p, dtype=np.float64)
    if max_sources is None:
        max_sources = int(np.diff(row_off).max()) if row_off.size > 1 else 0
    corpus = _Corpus(int(words.shape[0]), int(doc_group.shape[0]), int(vocab), words.ctypes.data,
                     doc_offsets.ctypes.data, int(init_seed) & (2**64 - 1),
                     None if hip_stream is None else int(hip_stream))
    groups = _Groups(int(n_groups), doc_group.ctypes.data)
    assoc = _Assoc(int(max_sources), row_off.ctypes.data, src.ctypes.data, p.ctypes.data)
    h = C.c_void_p()
    _check(lib().spdp_create_assoc(C.byref(corpus), C.byref(groups), C.byref(assoc), int(K),
                                   float(alpha), float(a), float(b), float(gamma), C.byref(h)))
    return h


def spdp_get_slots(h, slot_out):
    _check(lib().spdp_get_slots(h, _buf(slot_out)[0], _where(slot_out)))


def spdp_set_assignments_assoc(h, z, r, slot):
    if isinstance(z, np.ndarray):
        z = np.ascontiguousarray(z, dtype=np.int32)
        r = np.ascontiguousarray(r, dtype=np.uint8)
        slot = np.ascontiguousarray(slot, dtype=np.uint8)
    where = _where(z, r, slot)
    _check(lib().spdp_set_assignments_assoc(h, _buf(z)[0], _buf(r)[0], _buf(slot)[0], where))


def spdp_max_sources(h) -> int:
    S = C.c_int32()
    _check(lib().spdp_max_sources(h, C.byref(S)))
    return int(S.value)


def spdp_sweep(h, sweep: int, seed: int):
    _check(lib().spdp_sweep(h, int(sweep) & 0xFFFFFFFF, int(seed) & (2**64 - 1)))


def spdp_sweep_async(h, sweep: int, seed: int, waves: int = 0, live_totals: bool = False):
    _check(lib().spdp_sweep_async(h, int(sweep) & 0xFFFFFFFF, int(seed) & (2**64 - 1),
                                  int(waves), 1 if live_totals else 0))


def spdp_counts(h, g_begin, g_end, n_out=None, t_out=None):
    where = _where(n_out, t_out)
    _check(lib().spdp_counts(h, int(g_begin), int(g_end), _buf(n_out)[0], _buf(t_out)[0], where))


def spdp_totals(h, N_gk=None, T_gk=None, B_wk=None, B_k=None):
    where = _where(N_gk, T_gk, B_wk, B_k)
    _check(lib().spdp_totals(h, _buf(N_gk)[0], _buf(T_gk)[0], _buf(B_wk)[0], _buf(B_k)[0], where))


def spdp_loglik(h) -> float:
    out = C.c_double()
    _check(lib().spdp_loglik(h, C.byref(out)))
    return float(out.value)


def spdp_destroy(h):
    if h:
        lib().spdp_destroy(h)


def spdp_get_assignments(h, z_out=None, r_out=None):
    where = _where(z_out, r_out)
    _check(lib().spdp_get_assignments(h, _buf(z_out)[0], _buf(r_out)[0], where))


def spdp_set_assignments(h, z, r):
    if isinstance(z, np.ndarray):
        z = np.ascontiguousarray(z, dtype=np.int32)
        r = np.ascontiguousarray(r, dtype=np.uint8)
    where = _where(z, r)
    _check(lib().spdp_set_assignments(h, _buf(z)[0], _buf(r)[0], where))


def spdp_debug_conditionals(h, sweep, seed, tok_begin, tok_end, w_out=None, u_out=None,
                            zr_out=None):
    where = _where(w_out, u_out, zr_out)
    _check(lib().spdp_debug_conditionals(h, int(sweep) & 0xFFFFFFFF, int(seed) & (2**64 - 1),
                                         int(tok_begin), int(tok_end), _buf(w_out)[0],
                                         _buf(u_out)[0], _buf(zr_out)[0], where))


def spdp_stats(h):
    c, r = C.c_int64(), C.c_int64()
    _check(lib().spdp_stats(h, C.byref(c), C.byref(r)))
    return int(c.value), int(r.value)


def spdp_kernel_timing(h, enable: bool):
    _check(lib().spdp_kernel_timing(h, 1 if enable else 0))


def spdp_kernel_times(h):
    ms = np.zeros(SPDP_NKERNELS, dtype=np.float64)
    n = np.zeros(SPDP_NKERNELS, dtype=np.int64)
    _check(lib().spdp_kernel_times(h, ms.ctypes.data, n.ctypes.data))
    return {k: (float(ms[i]), int(n[i])) for i, k in enumerate(KERNEL_CLASSES)}


def spdp_read_probe(buf_ptr: int, nbytes: int, row_bytes: int = 0, rows: int = 0,
                    waves: int = 4096, stream=None) -> float:
    """Milliseconds to read a device buffer: whole (row_bytes = 0) or rows of
    row_bytes at pseudo-random positions, one row at a time per wavefront."""
    ms = C.c_double(0.0)
    _check(lib().spdp_read_probe(C.c_void_p(buf_ptr), int(nbytes), int(row_bytes), int(rows),
                                 int(waves), None if stream is None else C.c_void_p(int(stream)),
                                 C.byref(ms)))
    return ms.value


def spdp_hellinger_noalloc(h, p, q, out):
    """Device tensors p [V, kp], q [V, kq], out [kp, kq] (float64); enqueues
    only, on the state's stream."""
    V, kp = p.shape
    kq = q.shape[1]
    assert q.shape[0] == V and tuple(out.shape) == (kp, kq)
    for x in (p, q, out):
        assert x.is_cuda and x.dtype.is_floating_point and x.element_size() == 8
        assert x.is_contiguous()
    _check(lib().spdp_hellinger_noalloc(h, p.data_ptr(), kp, q.data_ptr(), kq, V,
                                        out.data_ptr()))


def spdp_check(h):
    """Number of failing cells, tokens and totals; raises SpdpError
    (SPDP_E_STATE) if there is any."""
    bad = C.c_int64(0)
    rc = lib().spdp_check(h, C.byref(bad))
    if rc == SPDP_E_STATE:
        raise SpdpError(rc, spdp_last_error())
    _check(rc)
    return int(bad.value)


def spdp_debug_poke(h, g, w, k, dn, dt):
    _check(lib().spdp_debug_poke(h, int(g), int(w), int(k), int(dn), int(dt)))


def spdp_info(h) -> dict:
    out = np.zeros(8, dtype=np.int64)
    _check(lib().spdp_info(h, out.ctypes.data))
    keys = ("N", "D", "V", "G", "K", "Kp", "ncap", "device_bytes")
    return {k: int(v) for k, v in zip(keys, out)}


def spdp_estimates(h, g_begin, g_end, theta=None, phi0=None, phi=None):
    where = _where(theta, phi0, phi)
    _check(lib().spdp_estimates(h, int(g_begin), int(g_end), _buf(theta)[0], _buf(phi0)[0],
                                _buf(phi)[0], where))


def spdp_heldout(h, words, doc_offsets, doc_group, n_groups, vocab, n_sweeps, seed, z_out=None):
    """(perplexity, sum of log p) of held-out documents; see include/spdp.h."""
    words = np.ascontiguousarray(words, dtype=np.int32)
    doc_offsets = np.ascontiguousarray(doc_offsets, dtype=np.int64)
    doc_group = np.ascontiguousarray(doc_group, dtype=np.int32)
    corpus = _Corpus(int(words.shape[0]), int(doc_group.shape[0]), int(vocab), words.ctypes.data,
                     doc_offsets.ctypes.data, 0, None)
    groups = _Groups(int(n_groups), doc_group.ctypes.data)
    out = np.zeros(2, dtype=np.float64)
    where = _where(z_out)
    _check(lib().spdp_heldout(h, C.byref(corpus), C.byref(groups), int(n_sweeps),
                              int(seed) & (2**64 - 1), out.ctypes.data, _buf(z_out)[0], where))
    return float(out[0]), float(out[1])


def spdp_hellinger(h, p, q, out):
    """Hellinger distances out [kp, kq] between the columns of p [V, kp] (None:
    the state's phi0) and q [V, kq]; see include/spdp.h."""
    where = _where(p, q, out)
    V, kq = q.shape
    kp = out.shape[0]
    if out.shape != (kp, kq) or (p is not None and p.shape != (V, kp)):
        raise ValueError("p [V, kp], q [V, kq] and out [kp, kq] do not agree")
    _check(lib().spdp_hellinger(h, _buf(p)[0], int(kp), _buf(q)[0], int(kq), int(V),
                                _buf(out)[0], where))
    return out


def spdp_align_topics(dist):
    """(match [kp] int32, total) of the least-total matching of rows to columns."""
    dist = np.ascontiguousarray(dist, dtype=np.float64)
    kp, kq = dist.shape
    match = np.zeros(kp, dtype=np.int32)
    total = C.c_double()
    _check(lib().spdp_align_topics(dist.ctypes.data, int(kp), int(kq), match.ctypes.data,
                                   C.byref(total)))
    return match, float(total.value)


# ---------------------------------------------------------------------------
# Convenience wrapper (host numpy in and out)
# ---------------------------------------------------------------------------
class Sampler:
    """Owns one library state; thin host-side helpers around the entry points."""

    def __init__(self, words, doc_offsets, doc_group, n_groups, vocab, K, alpha, a, b, gamma,
                 init_seed=0, hip_stream=None, assoc=None):
        """assoc: None (P = I) or (row_off, src, p) of the word associations."""
        if assoc is None:
            self.h = spdp_create(words, doc_offsets, doc_group, n_groups, vocab, K, alpha, a, b,
                                 gamma, init_seed, hip_stream)
        else:
            row_off, src, p = assoc
            self.h = spdp_create_assoc(words, doc_offsets, doc_group, n_groups, vocab, K, alpha,
                                       a, b, gamma, row_off, src, p, init_seed=init_seed,
                                       hip_stream=hip_stream)
        self.info = spdp_info(self.h)
        self.N, self.G, self.V, self.K = (self.info["N"], self.info["G"], self.info["V"],
                                          self.info["K"])
        self.S = spdp_max_sources(self.h)

    def close(self):
        if self.h:
            spdp_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def sweep(self, sweep, seed):
        spdp_sweep(self.h, sweep, seed)

    def sweep_async(self, sweep, seed, waves=0, live_totals=False):
        """The thesis's asynchronous sweep (an ablation; see include/spdp.h)."""
        spdp_sweep_async(self.h, sweep, seed, waves, live_totals)

    def assignments(self):
        z = np.empty(self.N, dtype=np.int32)
        r = np.empty(self.N, dtype=np.uint8)
        spdp_get_assignments(self.h, z, r)
        return z, r

    def set_assignments(self, z, r, slot=None):
        if slot is None:
            spdp_set_assignments(self.h, z, r)
        else:
            spdp_set_assignments_assoc(self.h, z, r, slot)

    def slots(self):
        """Source slot of each token's table (word associations; 0 for r = 0)."""
        s = np.empty(self.N, dtype=np.uint8)
        spdp_get_slots(self.h, s)
        return s

    def counts(self, g_begin=0, g_end=None):
        """n, t as [g][k][w] int32 arrays."""
        g_end = self.G if g_end is None else g_end
        n = np.empty((g_end - g_begin, self.K, self.V), dtype=np.int32)
        t = np.empty_like(n)
        spdp_counts(self.h, g_begin, g_end, n, t)
        return n, t

    def totals(self):
        N = np.empty((self.G, self.K), dtype=np.int32)
        T = np.empty_like(N)
        B = np.empty((self.V, self.K), dtype=np.int32)
        Bk = np.empty(self.K, dtype=np.int32)
        spdp_totals(self.h, N, T, B, Bk)
        return N, T, B, Bk

    def loglik(self):
        return spdp_loglik(self.h)

    def check(self):
        return spdp_check(self.h)

    def poke(self, g, w, k, dn, dt):
        spdp_debug_poke(self.h, g, w, k, dn, dt)

    def conditionals(self, sweep, seed, tok_begin, tok_end):
        T = tok_end - tok_begin
        per_topic = 2 if self.S == 0 else self.S + 1
        w = np.zeros((T, per_topic * self.K), dtype=np.float32)
        u = np.zeros(T, dtype=np.float32)
        zr = np.zeros(T, dtype=np.int32)
        spdp_debug_conditionals(self.h, sweep, seed, tok_begin, tok_end, w, u, zr)
        return w, u, zr

    def sampled(self, sweep, seed, tok_begin=0, tok_end=None):
        """Packed 2z + r of the sampling step only (before update and repair)."""
        tok_end = self.N if tok_end is None else tok_end
        zr = np.zeros(tok_end - tok_begin, dtype=np.int32)
        spdp_debug_conditionals(self.h, sweep, seed, tok_begin, tok_end, None, None, zr)
        return zr

    def stats(self):
        return spdp_stats(self.h)

    def estimates(self, g_begin=0, g_end=None):
        """(theta [D, K], phi0 [V, K], phi [g, V, K]) in fp64."""
        g_end = self.G if g_end is None else g_end
        theta = np.empty((self.info["D"], self.K), dtype=np.float64)
        phi0 = np.empty((self.V, self.K), dtype=np.float64)
        phi = np.empty((g_end - g_begin, self.V, self.K), dtype=np.float64)
        spdp_estimates(self.h, g_begin, g_end, theta, phi0, phi)
        return theta, phi0, phi

    def hellinger(self, q, p=None):
        """Hellinger distances [kp, kq] between the columns of p [V, kp] (default:
        this state's phi0) and q [V, kq], fp64 host arrays."""
        q = np.ascontiguousarray(q, dtype=np.float64)
        if p is not None:
            p = np.ascontiguousarray(p, dtype=np.float64)
        kp = self.K if p is None else p.shape[1]
        out = np.empty((kp, q.shape[1]), dtype=np.float64)
        return spdp_hellinger(self.h, p, q, out)

    def heldout(self, words, doc_offsets, doc_group, n_sweeps, seed):
        """(perplexity, sum of log p, fold-in topics) of held-out documents."""
        z = np.empty(len(words), dtype=np.int32)
        ppl, ll = spdp_heldout(self.h, words, doc_offsets, doc_group, self.G, self.V, n_sweeps,
                               seed, z)
        return ppl, ll, z
