"""Coefficients of the logistic GELU of the GEMM epilogue (common.h,
gelu_logistic).

GELU(u) = u Phi(u) with Phi(u) = sigma(g(u)), g an odd polynomial of degree 9.
g is the weighted least-squares fit to the logit of the standard normal CDF,
log(Phi / (1 - Phi)), on 40001 points of [-8, 8], with weights Phi (1 - Phi)
(the derivative of sigma, which carries an error in g into Phi).  The kernel
evaluates sigma(g) as 1 / (1 + 2^t), t = -g(u) log2(e), so the printed
coefficients are those of t in powers of u^2, times u.

Run: python fit_gelu_logistic.py  (numpy, scipy)."""
import numpy as np
from scipy.special import ndtr


def fit(deg=9, lo=-8.0, hi=8.0, n=40001):
    u = np.linspace(lo, hi, n)
    phi = ndtr(u)
    logit = np.log(phi) - np.log1p(-phi)
    w = phi * (1.0 - phi)
    powers = np.arange(1, deg + 1, 2)
    a = np.stack([u ** p for p in powers], 1)
    coef, *_ = np.linalg.lstsq(a * w[:, None], logit * w, rcond=None)
    return coef


if __name__ == "__main__":
    c = fit()
    t = -c / np.log(2.0)
    print("g(u) coefficients of u^1, u^3, ..., u^9:", " ".join("%.9e" % v for v in c))
    print("t(u) = u * P(u^2), P coefficients of (u^2)^0 .. (u^2)^4:", " ".join("%.9e" % v for v in t))
