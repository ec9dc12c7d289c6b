"""Coefficients of the polynomial the scoring kernel uses for the Shannon term.

The kernel sums the terms in base-2 units: with y = e / ln 2 it forms
g(1 + e) / ln 2 = y^2 psi(y), where g(u) = u log u - u + 1 and
psi(y) = ln 2 phi(y ln 2), phi(e) = g(1 + e) / e^2.  psi is taken on
|y| <= (1/4) / ln 2 (|e| <= 1/4) as a degree-5 polynomial in y: the Chebyshev
interpolant at 2000 Chebyshev nodes (fp64), converted to monomial
coefficients.  Prints the coefficients and the maximum relative error of psi
over the interval (fp64 evaluation, then fp32 Horner with fused
multiply-adds).  Only numpy is needed.
"""
import numpy as np
from numpy.polynomial import chebyshev

LN2 = np.log(2.0)
A = 0.25 / LN2    # half-width of the interval in y
DEG = 5


def phi(e):
    e = np.asarray(e, np.float64)
    out = np.empty_like(e)
    small = np.abs(e) < 1e-3
    k = np.arange(2, 40)
    out[small] = ((-e[small][:, None]) ** (k - 2) / (k * (k - 1))).sum(1)
    eb = e[~small]
    out[~small] = ((1 + eb) * np.log1p(eb) - eb) / eb ** 2
    return out


def psi(y):
    return LN2 * phi(LN2 * np.asarray(y, np.float64))


def fit():
    nodes = np.cos(np.pi * (np.arange(2000) + 0.5) / 2000) * A
    cheb = chebyshev.chebfit(nodes / A, psi(nodes), DEG)
    return chebyshev.cheb2poly(cheb) / A ** np.arange(DEG + 1)


if __name__ == "__main__":
    p = fit()
    grid = np.linspace(-A, A, 200001)
    ref = psi(grid)
    err64 = np.max(np.abs(np.polyval(p[::-1], grid) - ref) / ref)
    acc = np.full(grid.size, np.float32(p[-1]))
    g32 = grid.astype(np.float32)
    for c in p[-2::-1]:
        acc = (acc.astype(np.float64) * g32 + np.float64(np.float32(c))).astype(np.float32)
    err32 = np.max(np.abs(acc - ref) / ref)
    for i, c in enumerate(p):
        print("c%d = %.9e" % (i, c))
    print("interval |y| <= %.9e" % A)
    print("max relative error: fp64 %.2e, fp32 Horner %.2e" % (err64, err32))
