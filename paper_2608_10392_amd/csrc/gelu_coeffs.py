"""Coefficients of the bf16 up-projection's GELU (common.hpp, gelu_exp2poly).

GELU(x) = x Phi(x) = max(x, 0) - |x| Phi(-|x|), and Phi(-y) = 2^Q(y) with
Q(y) = log2 Phi(-y), a smooth function on y >= 0 (Q(0) = -1, about
-y^2 / (2 ln 2) for large y). Q is fitted on [0, Y] by a degree-D polynomial
(least squares in the Chebyshev basis on 20,001 points, then expanded into
powers of y); the kernel evaluates it by Horner's rule in fp32 at
min(|x|, Y). Printed as the C initialiser used in common.hpp.

Run: python paper_2608_10392_amd/csrc/gelu_coeffs.py
"""
import numpy as np
from scipy.special import log_ndtr

Y, D = 6.0, 7


def coefficients(y_max=Y, degree=D):
    y = np.linspace(0.0, y_max, 20001)
    q = log_ndtr(-y) / np.log(2.0)
    cheb = np.polynomial.chebyshev.chebfit(2.0 * y / y_max - 1.0, q, degree)
    in_t = np.polynomial.Polynomial(np.polynomial.chebyshev.cheb2poly(cheb))
    in_y = in_t(np.polynomial.Polynomial([-1.0, 2.0 / y_max]))
    return [float(np.float32(c)) for c in in_y.coef]


if __name__ == "__main__":
    c = coefficients()
    print(f"// Q(y) = sum c[i] y^i, i = 0..{D}, fitted on [0, {Y:g}]")
    print("constexpr float kGeluQ[%d] = {%s};" % (len(c), ", ".join("%.9ef" % v for v in c)))
