"""Coefficients of the branch-free GELU in ks_epilogue.h (gelu_f32).

GELU(x) = x Phi(x) with Phi the standard normal CDF.  For z = |x| / sqrt 2 the
lower tail is Phi(-|x|) = erfc(z) / 2, and with u = 1 / (2 + z) in (0, 1/2]

    erfc(z) / 2 = u * 2^(-log2(e) x^2 / 2 + R(u)),  R(u) = log2(erfcx(z) / (2 u)),

where erfcx(z) = exp(z^2) erfc(z).  R is smooth on the whole interval (it tends
to -log2(2 sqrt(pi)) as u -> 0), so a low-degree polynomial fits it to near
single precision.  This script fits R by Chebyshev interpolation over
|x| <= 16 (beyond which x Phi(-|x|) underflows in fp32) and prints the
monomial coefficients R(u) = sum_k C[k] u^k as float literals: degree 9 for
fp32 outputs, degree 5 for 16-bit outputs.

Run: python gelu_fit.py   (numpy + scipy; writes nothing)
"""
import numpy as np
from scipy.special import erfcx

DEGREE = 9          # fp32 outputs (kGeluR*)
DEGREE_16BIT = 5    # 16-bit outputs (kGeluS*)
XMAX = 16.0
NODES = 800


def r_exact(u):
    z = 1.0 / u - 2.0
    return np.log2(erfcx(z) / (2.0 * u))


def fit(degree=DEGREE):
    lo, hi = 1.0 / (2.0 + XMAX / np.sqrt(2.0)), 0.5
    s = np.cos(np.pi * (np.arange(NODES) + 0.5) / NODES)
    cheb = np.polynomial.chebyshev.chebfit(s, r_exact(lo + (hi - lo) * (s + 1) / 2), degree)
    in_s = np.polynomial.chebyshev.cheb2poly(cheb)
    # s = (2u - (lo + hi)) / (hi - lo)
    s_of_u = np.polynomial.polynomial.Polynomial([-(lo + hi) / (hi - lo), 2.0 / (hi - lo)])
    coef = np.polynomial.polynomial.Polynomial(in_s)(s_of_u).coef
    u = np.linspace(lo, hi, 100001)
    err = np.max(np.abs(np.polynomial.polynomial.polyval(u, coef.astype(np.float32).astype(np.float64)) - r_exact(u)))
    return coef.astype(np.float32), err


if __name__ == "__main__":
    for degree, name in ((DEGREE, "kGeluR"), (DEGREE_16BIT, "kGeluS")):
        c, err = fit(degree)
        print("// degree %d: max |R_fit - R| over |x| <= %g: %.2e (log2 units)" % (degree, XMAX, err))
        for k, v in enumerate(c):
            print("constexpr float %s%d = %.9gf;" % (name, k, v))
