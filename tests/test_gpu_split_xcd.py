"""Split-K partials exchanged through one XCD's L2, and the fallback when a
chunk is not on the XCD that round-robin dispatch gives it.

Every chunk that finds itself off its expected XCD writes its partial through
to memory and flags its arrival; the readers then fetch that partial from
memory and, when a tile's chunks are mixed, one chunk on the expected XCD
finishes the whole tile.  The additions are the same in every case, so the
output bits must not depend on which chunks are foreign.  Real dispatch puts
every chunk where expected, so the test forces the fallback with
NJ_TEST_SPLIT_FOREIGN (a bit mask of chunks that act as foreign) in child
processes, one per mask, and compares the output digests bitwise."""
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))


def _run(mask):
    env = dict(os.environ)
    if mask is not None:
        env["NJ_TEST_SPLIT_FOREIGN"] = hex(mask)
    print(f"split-K foreign-chunk child, mask={mask}", flush=True)
    r = subprocess.run([sys.executable, "-u", os.path.join(HERE, "_split_foreign_child.py")], env=env,
                       capture_output=True, text=True, timeout=240)
    assert r.returncode == 0, r.stderr[-3000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.startswith("case ")]
    assert len(lines) == 6, r.stdout
    return lines


def test_split_partials_same_bits_whatever_chunks_are_foreign():
    base = _run(None)
    for ln in base:
        assert "err=0" in ln and "repeat_same=True" in ln, ln
    for mask in (0x1, 0x2, 0x5, 0xff):  # one foreign chunk (first / second), several, all
        got = _run(mask)
        for b, g in zip(base, got):
            assert "err=0" in g and "repeat_same=True" in g, (mask, g)
            assert g == b, (mask, b, g)
