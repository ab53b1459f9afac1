"""Closed forms the paper states, used to pin the oracle.

TEST INFRASTRUCTURE ONLY (see the package docstring).

* Rate of the union of k Voronoi codes of nesting ratio q in dimension 8 (Sec. 3,
  "Overload avoidance via union of Voronoi codes"): log2(q) + log2(k) / 8 bits per entry.
* The lower bound on the inner-product distortion of rate-R quantizers for iid Gaussian
  vectors (Sec. 2.1, eqs. lbnd and gammadef): E (X^T Y - est)^2 >= n Gamma(R).  Below
  R* the bound is the straight line from (0, 1) that touches the curve
  2 * 2^(-2R) - 2^(-4R); R* is the touching point (the paper quotes R* ~ 0.906).
* The normalized second moment of E8 (Sec. 3): 929 / 12960 ~ 0.0716821 (Conway & Sloane's
  closed form of the value the paper quotes).
"""

import math

NSM_E8 = 929.0 / 12960.0


def rate_bits(q, k):
    return math.log2(q) + math.log2(k) / 8.0


def _phi(R):
    return 2.0 * 2.0 ** (-2.0 * R) - 2.0 ** (-4.0 * R)


def _dphi(R):
    ln2 = math.log(2.0)
    return -4.0 * ln2 * 2.0 ** (-2.0 * R) + 4.0 * ln2 * 2.0 ** (-4.0 * R)


def r_star():
    """Touching point of the line through (0, 1): (phi(R) - 1) / R = phi'(R), by bisection."""
    lo, hi = 0.1, 3.0
    f = lambda R: (_phi(R) - 1.0) / R - _dphi(R)  # noqa: E731
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        if (f(lo) < 0) == (f(mid) < 0):
            lo = mid
        else:
            hi = mid
    return 0.5 * (lo + hi)


def gamma(R):
    Rs = r_star()
    if R >= Rs:
        return _phi(R)
    return 1.0 - (1.0 - _phi(Rs)) * R / Rs
