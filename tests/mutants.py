"""Planted mistakes in the oracle (no tests in this module).

A mutant is oracle.c with one textual edit inside one function, compiled into
a library of its own in a temporary directory.  The pins of the oracle must
fail on every mutant listed next to them: that is how a test shows it would
catch a plausible slip of the oracle (a dropped update, a wrong index, live
instead of snapshot counts).  Mutants are built and run on the CPU only.
"""
from __future__ import annotations

import os
import re
import subprocess
import tempfile

import oracle

_SRC = os.path.join(os.path.dirname(os.path.abspath(oracle.__file__)), "oracle.c")


def mutant_source(function: str, old: str, new: str) -> str:
    """oracle.c with the first `old` after the definition of `function`
    replaced by `new` (the edit must fall inside that function)."""
    src = open(_SRC).read()
    start = -1
    for mt in re.finditer(rf"^[A-Za-z_].*\b{re.escape(function)}\(", src, re.MULTILINE):
        # a definition (its body opens before any semicolon), not a prototype
        brace, semi = src.find("{", mt.end()), src.find(";", mt.end())
        if brace >= 0 and (semi < 0 or brace < semi):
            start = mt.start()
            break
    assert start >= 0, f"no definition of {function}"
    end = src.find("\n}\n", start)
    pos = src.find(old, start)
    assert 0 <= pos < end, f"{old!r} not found inside {function}"
    return src[:pos] + new + src[pos + len(old):]


class Mutant:
    """Build the mutant library; use it as `with oracle.swap_library(mut.path)`."""

    def __init__(self, function: str, old: str, new: str, prelude: str = ""):
        self._dir = tempfile.TemporaryDirectory(prefix="oracle_mutant_")
        src = mutant_source(function, old, new)
        if prelude:
            # declarations the edit needs, placed after the includes
            anchor = "#define OR_PURPOSE_SAMPLE"
            src = src.replace(anchor, prelude + "\n" + anchor, 1)
        c_path = os.path.join(self._dir.name, "oracle_mutant.c")
        self.path = os.path.join(self._dir.name, "liboracle_mutant.so")
        with open(c_path, "w") as f:
            f.write(src)
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", c_path, "-lm", "-o",
                               self.path])

    def close(self):
        self._dir.cleanup()

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()
        return False
