"""The e4m3 append's division-free quotient (CPU).

Appending to an e4m3 pool takes RN(x / s) for a scale s shared by a whole
(block, head) tile, as r = RN(1/s), q0 = RN(x r), then Markstein's
correction q1 = fma(fma(-q0, s, x), r, q0), with q0 kept past 512 (those
values saturate) and q0's sign; scales outside [2^-100, 2^100] divide.
`tests/csrc/e4m3_quotient_check.c` re-implements that sequence in C (IEEE
single precision with fmaf, no contraction) and compares the resulting e4m3
code, for every finite bf16 x, with the code of the correctly rounded
quotient, found by a plain nearest-value search.  Here every 16th scale
b / 448 (b a positive bf16) is taken, plus the edges of the fast range and 1;
the same program with stride 1 covers all 2.1e9 pairs (about 80 s)."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_division_free_quotient_gives_the_rounded_quotients_codes(tmp_path):
    exe = tmp_path / "qchk"
    subprocess.run(["gcc", "-O2", "-ffp-contract=off", "-o", str(exe),
                    os.path.join(HERE, "csrc", "e4m3_quotient_check.c"), "-lm"], check=True)
    out = subprocess.run([str(exe), "16"], capture_output=True, text=True, check=True).stdout
    pairs, bad = (int(v) for v in out.split()[-2:])
    assert pairs > 1.3e8 and bad == 0, out
