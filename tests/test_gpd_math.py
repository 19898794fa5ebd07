"""Host check of the library's fp64 GPD likelihood terms (csrc/gpd_math.h): a = t/(1+t) and
b = log1p(t) for t > -1, against correctly rounded references. The header is compiled for the
host with hipcc; nothing here touches a GPU."""
import math
import os
import shutil
import subprocess
import tempfile
from fractions import Fraction

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2407_09486_amd", "csrc")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"

PROGRAM = r"""
#include "gpd_math.h"
#include <cstdio>
int main() {
    double t;
    while (std::scanf("%lf", &t) == 1) {
        double a, b;
        enova::gpd_terms(t, a, b);
        std::printf("%a %a\n", a, b);
    }
    return 0;
}
"""


@pytest.fixture(scope="module")
def terms():
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    d = tempfile.mkdtemp()
    try:
        src = os.path.join(d, "t.cpp")
        exe = os.path.join(d, "t")
        with open(src, "w") as f:
            f.write(PROGRAM)
        subprocess.run([HIPCC, "-O2", "-x", "hip", "--offload-arch=gfx950", "-I", CSRC, src, "-o", exe],
                       check=True, capture_output=True)

        def run(ts):
            out = subprocess.run([exe], input="\n".join(repr(float(t)) for t in ts), text=True,
                                 capture_output=True, check=True).stdout.split("\n")
            ab = [line.split() for line in out if line.strip()]
            return (np.array([float.fromhex(p[0]) for p in ab]),
                    np.array([float.fromhex(p[1]) for p in ab]))
        yield run
    finally:
        shutil.rmtree(d, ignore_errors=True)


def _samples():
    rng = np.random.default_rng(7)
    ts = [0.0, 5e-324, 1e-300, 1e-20, -1e-20, 1e-10, -1e-10, 1e-5, 0.5, -0.5, 1.0, 2.0,
          -1.0 + 2.0 ** -52, -1.0 + 1e-10, -0.9999999999, math.sqrt(0.5) - 1.0, math.sqrt(2.0) - 1.0,
          1e30, 1e300, 3.5, 0.7, -0.3]
    ts += list(-np.expm1(-rng.exponential(3.0, 4000)))               # (-1, 0)
    ts += list(10.0 ** rng.uniform(-18, 18, 4000))                    # (0, 1e18)
    ts += list(rng.uniform(-0.4, 0.5, 2000))                          # around the reduction seams
    return np.array(ts, dtype=np.float64)


def test_log1p_within_three_ulp(terms):
    ts = _samples()
    _, b = terms(ts)
    ref = np.array([math.log1p(t) for t in ts])
    err = np.abs(b - ref)
    ulp = np.spacing(np.abs(ref))
    ok = (err <= 3 * ulp) | (ref == 0) & (b == 0)   # the rounded s = (m-1)/(m+1) costs up to ~2 ulp
    assert ok.all(), list(zip(ts[~ok][:5], b[~ok][:5], ref[~ok][:5]))


def test_ratio_within_two_ulp(terms):
    ts = _samples()
    a, _ = terms(ts)
    ref = np.array([float(Fraction(t) / (1 + Fraction(t))) for t in ts])
    err = np.abs(a - ref)
    assert (err <= 2 * np.spacing(np.abs(ref))).all()


def test_zero_and_sign(terms):
    a, b = terms([0.0, -0.25, 0.25])
    assert a[0] == 0.0 and b[0] == 0.0
    assert a[1] < 0 and b[1] < 0 and a[2] > 0 and b[2] > 0
