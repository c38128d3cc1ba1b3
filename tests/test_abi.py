"""The C ABI without a GPU: the library loads, exports every entry point that
include/spdp.h declares, and rejects invalid arguments before touching HIP."""
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_entry_points():
    src = open(os.path.join(ROOT, "include", "spdp.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(spdp_[a-z_0-9]+)\s*\(", src)))


def test_header_declares_the_boundary():
    names = declared_entry_points()
    for must in ("spdp_create", "spdp_sweep", "spdp_counts", "spdp_loglik", "spdp_destroy"):
        assert must in names


def test_library_exports_every_declared_symbol():
    from paper_1510_06549_amd import spdp as sp

    L = sp.lib()
    for name in declared_entry_points():
        assert hasattr(L, name), name
    assert sorted(sp.EXPORTS) == declared_entry_points()


def test_invalid_arguments_rejected_without_gpu():
    from paper_1510_06549_amd import spdp as sp

    words = np.array([0, 1, 2], np.int32)
    off = np.array([0, 3], np.int64)
    grp = np.array([0], np.int32)
    cases = [
        dict(K=0), dict(K=sp.SPDP_MAX_K + 1), dict(alpha=0.0), dict(alpha=float("nan")),
        dict(a=1.0), dict(a=-0.1), dict(b=0.0), dict(gamma=0.0),
    ]
    for kw in cases:
        args = dict(K=4, alpha=0.1, a=0.5, b=1.0, gamma=0.1)
        args.update(kw)
        with pytest.raises(sp.SpdpError) as e:
            sp.spdp_create(words, off, grp, 1, 3, args["K"], args["alpha"], args["a"], args["b"],
                           args["gamma"])
        assert e.value.code == sp.SPDP_E_ARG, kw
    # offsets that do not end at N, or decrease
    for bad_off in (np.array([0, 2], np.int64), np.array([1, 3], np.int64)):
        with pytest.raises(sp.SpdpError) as e:
            sp.spdp_create(words, bad_off, grp, 1, 3, 4, 0.1, 0.5, 1.0, 0.1)
        assert e.value.code == sp.SPDP_E_ARG
    with pytest.raises(sp.SpdpError) as e:
        sp.spdp_create(np.zeros(4, np.int32), np.array([0, 3, 2, 4], np.int64),
                       np.zeros(3, np.int32), 1, 3, 4, 0.1, 0.5, 1.0, 0.1)
    assert e.value.code == sp.SPDP_E_ARG
    # G * V too large
    with pytest.raises(sp.SpdpError) as e:
        sp.spdp_create(words, off, grp, 70000, 40000, 4, 0.1, 0.5, 1.0, 0.1)
    assert e.value.code == sp.SPDP_E_ARG
    assert "n_groups * vocab" in sp.spdp_last_error()


def test_null_state_is_an_argument_error():
    from paper_1510_06549_amd import spdp as sp

    L = sp.lib()
    assert L.spdp_sweep(None, 0, 0) == sp.SPDP_E_ARG
    assert L.spdp_stats(None, None, None) == sp.SPDP_E_ARG
    assert L.spdp_check(None, None) == sp.SPDP_E_ARG
    assert L.spdp_debug_poke(None, 0, 0, 0, 1, 0) == sp.SPDP_E_ARG
    L.spdp_destroy(None)  # NULL is ignored


def test_invalid_associations_rejected_without_gpu():
    from paper_1510_06549_amd import spdp as sp

    words = np.array([0, 1, 2], np.int32)
    off = np.array([0, 3], np.int64)
    grp = np.array([0], np.int32)
    V = 3

    def create(row_off, src, p, S=None):
        return sp.spdp_create_assoc(words, off, grp, 1, V, 2, 0.1, 0.5, 1.0, 0.1, row_off, src,
                                    p, max_sources=S)

    good = (np.array([0, 2, 3, 5]), np.array([0, 1, 1, 2, 0]), np.array([.5, .5, 1., .5, .5]))
    cases = [
        ((np.array([0, 2, 2, 4]), np.array([0, 1, 2, 0]), np.array([.5, .5, .5, .5])), None,
         "no source"),
        ((good[0], np.array([0, 1, 1, 2, 3]), good[2]), None, "out of [0, vocab)"),
        ((good[0], np.array([0, 0, 1, 2, 0]), good[2]), None, "repeats source"),
        ((good[0], good[1], np.array([.5, 0., 1., .5, .5])), None, "finite and > 0"),
        ((good[0], good[1], np.array([.5, np.inf, 1., .5, .5])), None, "finite and > 0"),
        (good, 3, "longest row"),
        (good, 9, "max_sources must be in"),
        ((np.array([0, 9, 10, 11]), np.arange(11) % 3, np.ones(11)), 9, "max_sources must be in"),
    ]
    for (ro, src, p), S, msg in cases:
        with pytest.raises(sp.SpdpError) as e:
            create(ro, src, p, S)
        assert e.value.code == sp.SPDP_E_ARG, msg
        assert msg in sp.spdp_last_error(), (msg, sp.spdp_last_error())
    L = sp.lib()
    assert L.spdp_create_assoc(None, None, None, 2, 0.1, 0.5, 1.0, 0.1, None) == sp.SPDP_E_ARG
    assert L.spdp_get_slots(None, None, 0) == sp.SPDP_E_ARG
    assert L.spdp_max_sources(None, None) == sp.SPDP_E_ARG


def test_read_probe_arguments_rejected_without_gpu():
    from paper_1510_06549_amd import spdp as sp

    bad = [
        dict(buf_ptr=0, nbytes=1 << 20),                              # NULL buffer
        dict(buf_ptr=16 * 1001 + 8, nbytes=1 << 20),                  # misaligned
        dict(buf_ptr=1 << 20, nbytes=1 << 20, row_bytes=512, rows=1),  # row size
        dict(buf_ptr=1 << 20, nbytes=8),                               # below 16 bytes
        dict(buf_ptr=1 << 20, nbytes=1024, row_bytes=2048, rows=1),    # below one row
        dict(buf_ptr=1 << 20, nbytes=1 << 20, waves=0),
        dict(buf_ptr=1 << 20, nbytes=1 << 20, row_bytes=1024, rows=0),
    ]
    for kw in bad:
        with pytest.raises(sp.SpdpError) as e:
            sp.spdp_read_probe(**kw)
        assert e.value.code == sp.SPDP_E_ARG, kw
