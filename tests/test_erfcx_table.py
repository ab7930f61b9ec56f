"""The erfcx coefficient table of the device's U-sampler and acceptance scan
(Weideman's rational approximation, erfcx_table.hpp): it is what its
generator writes, and evaluated in the device's form it reproduces
scipy.special.erfcx to the stated 1e-15 relative error on y >= 0."""
import pathlib
import re
import subprocess
import sys

import numpy as np
from scipy.special import erfcx

CSRC = pathlib.Path(__file__).resolve().parents[1] / "paper_2606_13426_amd" / "csrc"


def _table():
    s = (CSRC / "erfcx_table.hpp").read_text()
    L = float(re.search(r"kWeidemanL = ([^;]+);", s).group(1))
    a = [float(x) for x in re.findall(r"^\s+([-0-9.e+]+),$", s, re.M)]
    n = int(re.search(r"kWeidemanN = (\d+);", s).group(1))
    assert len(a) == n
    return L, np.array(a)


def test_table_matches_generator():
    out = subprocess.run([sys.executable, str(CSRC / "gen_erfcx_table.py")], capture_output=True,
                         text=True, check=True).stdout
    assert out == (CSRC / "erfcx_table.hpp").read_text()


def test_table_reproduces_erfcx():
    L, a = _table()
    y = np.concatenate([np.linspace(0.0, 12.0, 48001), np.logspace(-12, 19, 6000), [0.0, 1e300]])
    inv = 1.0 / (L + y)
    z = (L - y) * inv
    p = np.full_like(y, a[0])
    for c in a[1:]:
        p = p * z + c
    got = (2.0 * p * inv + 1.0 / np.sqrt(np.pi)) * inv
    ref = erfcx(y)
    assert np.all(np.abs(got - ref) <= 1e-15 * ref)
