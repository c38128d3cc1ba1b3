"""bench.py's argument handling on the host: every refusal exits with status 2
and a message before any device work (the measurement itself runs on a GPU)."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args],
                          capture_output=True, text=True, timeout=120)


@pytest.mark.parametrize("args,needle", [
    (("--gpus", "2"), "one GPU"),
    (("--gpus", "8", "--steps", "1"), "one GPU"),
    (("--heldout", "1"), "at least 2 fold-in sweeps"),
    (("--heldout", "10", "--async"), "not a sweep variant"),
    (("--async", "--assoc", "4"), "P = I only"),
])
def test_refusals(args, needle):
    p = _run(*args)
    assert p.returncode == 2, (p.returncode, p.stderr)
    assert needle in p.stderr
    assert p.stdout == ""
