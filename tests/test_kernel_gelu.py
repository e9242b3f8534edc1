"""The bf16 up-projection's GELU approximation (csrc/common.hpp, gelu_exp2poly).

Host-side check of the kernel's arithmetic: the coefficients in the header
are the ones the committed fit script prints, and the formula, evaluated in
fp32 steps here, stays within its stated error of x Phi(x) (scipy's normal
CDF in fp64). No GPU needed.
"""
import os
import re
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_10392_amd", "csrc")
special = pytest.importorskip("scipy.special")


def header_coefficients():
    text = open(os.path.join(CSRC, "common.hpp")).read()
    body = re.search(r"kGeluQ\[8\]\s*=\s*\{([^}]*)\}", text).group(1)
    ymax = float(re.search(r"kGeluQMax\s*=\s*([0-9.eE+-]+)f", text).group(1))
    return [float(v.strip().rstrip("f")) for v in body.split(",")], ymax


def f32(v):
    return np.asarray(v, dtype=np.float64).astype(np.float32).astype(np.float64)


def fma32(a, b, c):
    # fp32 operands: the product is exact in fp64, so this rounds once more
    # than a fused fp32 fma at most in rare halfway cases.
    return f32(np.asarray(a, np.float64) * b + c)


def gelu_kernel(x, c, ymax):
    """gelu_exp2poly in fp32 steps: Q evaluated at |x| (no clamp)."""
    x = f32(x)
    y = np.abs(x)
    q = fma32(c[7], y, c[6])
    for i in range(5, -1, -1):
        q = fma32(q, y, c[i])
    e = f32(np.exp2(q))
    return fma32(np.abs(x), f32(0.5 - e), f32(0.5 * x))


def test_header_matches_fit_script():
    sys.path.insert(0, CSRC)
    dont_write = sys.dont_write_bytecode
    sys.dont_write_bytecode = True   # no cache files beside the kernel sources
    try:
        import gelu_coeffs
    finally:
        sys.dont_write_bytecode = dont_write
        sys.path.pop(0)
    c, ymax = header_coefficients()
    assert ymax == gelu_coeffs.Y
    np.testing.assert_array_equal(np.float32(c), np.float32(gelu_coeffs.coefficients()))


def test_error_bounds():
    c, ymax = header_coefficients()
    x = np.concatenate([np.linspace(-12, 12, 480001), [0.0, 1e-30, -1e-30, 1e-6, -1e-6, 6.0, -6.0]])
    x = f32(x)
    exact = x * special.ndtr(x)
    got = gelu_kernel(x, c, ymax)
    err = np.abs(got - exact)
    assert err.max() < 5e-7
    # Relative 1e-5 from the fit, plus the rounding of 1/2 - Phi(-|a|) to
    # fp32 (at most 2^-25 |a|), which dominates in the far negative tail.
    inside = np.abs(x) < ymax
    assert (err[inside] <= 1e-5 * np.abs(exact[inside]) + 3e-8 * np.abs(x[inside])).all()
    pos = x > -2
    assert (err[pos] <= 1e-5 * np.abs(exact[pos])).all()
    # GELU(0) = 0 and the signs of the two branches.
    assert gelu_kernel(np.array([0.0]), c, ymax)[0] == 0.0
    assert (got[x > 0] > 0).all() and (got[x < 0] <= 0).all()


def test_polynomial_falls_past_the_fit_range():
    """The forward evaluates Q at |x| without clamping: past the fit range
    the fp32 Horner value must stay at or below Q(Y) (so 2^Q <= Phi(-Y)-sized
    values) and reach -inf for huge |x|."""
    c, ymax = header_coefficients()
    y = f32(np.concatenate([np.linspace(ymax, 200.0, 200001), np.geomspace(200.0, 3e38, 4000)]))
    with np.errstate(over="ignore", invalid="ignore"):
        q = fma32(c[7], y, c[6])
        for i in range(5, -1, -1):
            q = fma32(q, y, c[i])
    assert (q <= q[0]).all() and q[0] < -29.0
    assert np.all(np.diff(q[np.isfinite(q)]) <= 0)
    assert q[-1] == -np.inf


def test_infinities_and_nan():
    c, ymax = header_coefficients()
    with np.errstate(invalid="ignore"):
        v = gelu_kernel(np.array([np.inf, np.nan]), c, ymax)
    assert v[0] == np.inf and np.isnan(v[1])


def gelu_grad_kernel(x, c, ymax):
    """gelu_exp2poly_grad's derivative in fp32 steps: the fitted
    Phi(-|x|) = 2^Q(|x|) gives Phi(x), and phi(x) = 2^(-x^2 log2(e)/2) / sqrt(2 pi)."""
    x = f32(x)
    y = np.minimum(np.abs(x), ymax)
    q = fma32(c[7], y, c[6])
    for i in range(5, -1, -1):
        q = fma32(q, y, c[i])
    P = f32(np.exp2(q))
    Phi = np.where(x >= 0, f32(1.0 - P), P)
    phi2 = f32(np.exp2(f32(f32(np.float32(-0.7213475204444817) * x) * x)))
    return fma32(f32(x * np.float32(0.3989422804014327)), phi2, Phi)


def test_derivative_error_bound():
    """d GELU/dx = Phi(x) + x phi(x) within 5e-6 (absolute) of the exact
    derivative everywhere, as the header states; the backward rounds it to
    fp16 (spacing 2^-11 near 1) right after."""
    c, ymax = header_coefficients()
    x = f32(np.concatenate([np.linspace(-14, 14, 560001), [0.0, 1e-30, -1e-30, 6.0, -6.0, 40.0, -40.0]]))
    exact = special.ndtr(x) + x * np.exp(-0.5 * x * x) / np.sqrt(2.0 * np.pi)
    got = gelu_grad_kernel(x, c, ymax)
    assert np.abs(got - exact).max() < 5e-6
    # the limits: 1 for large x, 0 for very negative x, 1/2 at 0 (to the fit)
    assert abs(gelu_grad_kernel(np.array([40.0]), c, ymax)[0] - 1.0) < 1e-8
    assert abs(gelu_grad_kernel(np.array([-40.0]), c, ymax)[0]) < 1e-8
    assert abs(gelu_grad_kernel(np.array([0.0]), c, ymax)[0] - 0.5) < 5e-6


def test_derivative_matches_header_formula():
    """The constants the host model uses are the ones in the header."""
    text = open(os.path.join(CSRC, "common.hpp")).read()
    body = text[text.index("void gelu_exp2poly_grad"):]
    body = body[:body.index("\n}\n")]
    assert "-0.7213475204444817f" in body and "0.3989422804014327f" in body
    assert "a >= 0.0f ? 1.0f - P : P" in body
