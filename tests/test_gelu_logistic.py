"""Pin of the GEMM epilogue's logistic GELU (common.h, gelu_logistic).

The coefficients are read from the source and the formula is evaluated in
fp32, as the kernel does: t = u P(u^2), GELU = u / (1 + 2^t).  It is held
against the exact u Phi(u) (scipy's normal CDF, float64) over the fit range
and far past it.  It is also held against the fit script's output, so that a
coefficient typed wrong fails here."""
import os
import re
import subprocess
import sys

import numpy as np
from scipy.special import ndtr

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2502_19864_amd", "csrc")


def _coefficients():
    src = open(os.path.join(CSRC, "common.h")).read()
    body = src[src.index("float gelu_logistic(float u)"):]
    body = body[:body.index("\n}\n")]
    nums = [float(v) for v in re.findall(r"([-+]?\d\.\d+e[-+]\d+)f", body)]
    # fmaf(x2, c4, c3), then c2, c1, c0: P coefficients of (u^2)^4 .. (u^2)^0
    assert len(nums) == 5, nums
    return np.array(nums, dtype=np.float64)


def _gelu_f32(u, c):
    u = u.astype(np.float32)
    c = c.astype(np.float32)  # c4, c3, c2, c1, c0
    x2 = u * u
    p = x2 * c[0] + c[1]
    for k in (2, 3, 4):
        p = p * x2 + c[k]
    t = (p * u).astype(np.float64)
    with np.errstate(over="ignore"):
        e = np.exp2(t).astype(np.float32)
        return u * (np.float32(1) / (np.float32(1) + e))


def test_coefficients_match_the_fit():
    c = _coefficients()  # c4 .. c0
    out = subprocess.run([sys.executable, os.path.join(CSRC, "fit_gelu_logistic.py")], capture_output=True,
                         text=True, check=True).stdout
    line = [l for l in out.splitlines() if l.startswith("t(u)")][0]
    fit = np.array([float(v) for v in line.split(":")[1].split()])  # c0 .. c4
    assert np.allclose(c[::-1], fit, rtol=1e-6, atol=0), (c[::-1], fit)


def test_error_bound_over_the_real_line():
    c = _coefficients()
    u = np.concatenate([np.linspace(-30, 30, 600001), [-1e4, -100.0, 100.0, 1e4]])
    got = _gelu_f32(u, c).astype(np.float64)
    ref = u * ndtr(u)
    err = np.abs(got - ref)
    assert np.all(np.isfinite(got))
    assert err.max() <= 7e-6, err.max()
    # relative to the value where it is not tiny: far below bf16's 2^-9
    big = np.abs(ref) > 1e-2
    assert (err[big] / np.abs(ref[big])).max() < 2e-4
    # the limits: 0 far left, u far right
    assert got[-4] == 0.0 and abs(got[-1] - 1e4) < 1e-3
