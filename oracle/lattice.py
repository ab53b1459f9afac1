"""Gosset lattice E8: generator of 2E8 and the nearest-point map Q_E8.

TEST INFRASTRUCTURE ONLY (see the package docstring): the product path never uses this.

Paper passages followed:

* Sec. 3 "Lattices", eq. (QLdef): Q_Lambda(x) = argmin over lattice points of ||x - lambda||,
  ties broken in a fixed, systematic way.
* Sec. 4.1 and App. C: E8 = D8 u (D8 + 1/2), where D8 is the set of integer vectors with
  an even coordinate sum; the nearest point is the closer of the nearest D8 point and the
  nearest D8+1/2 point (Conway and Sloane).
* App. C, Alg. 5 ("Oracle for the Gosset lattice"): round down to d, decide per coordinate
  whether to round up (g), fix the parity of each candidate by moving the single coordinate
  whose move costs least, and keep the candidate with the smaller squared distance.
* App. E: the generator G of 2E8 (not E8), so that lattice points are integer vectors.
* App. D (NestQuantM): a decoder-side variant f of the oracle that fixes the parity of both
  candidates at the first coordinate instead of at argmax / argmin (``nearest_e8_m_rational``).

Points are carried in "2E8 units": a point p of E8 is stored as the integer vector P = 2p.

Readings of Alg. 5 (the printed listing is garbled in two places):

1. D8 parity fix.  Moving coordinate i of the D8 candidate to the other neighbouring
   integer raises its squared error from e_i^2 to (1 - e_i)^2, by 1 - 2 e_i, where e_i is
   the distance of y_i to the nearest integer.  The cheapest move is at argmax e.  The
   D8-minus-(D8+1/2) gap therefore grows by 1 - 2 e_p.  (The printed update of Delta for
   this branch has the wrong form; the derivation in App. C and the paper's own decoder
   listing in App. E both give this one.)
2. D8+1/2 parity fix.  Moving coordinate i of the half-integer candidate to the other
   neighbouring half-integer raises its squared error by 2 e_i; the cheapest move is at
   argmin e, and it moves towards y (up when y_i lies above d_i + 1/2, else down).
3. Ties, all broken "systematically" (Sec. 3): an exact half rounds down (g is a strict
   comparison), argmax / argmin take the lowest index, and an exact tie between the two
   candidates returns the D8+1/2 candidate (Alg. 5 returns the D8 point only when
   Delta > 2 strictly).
4. The D8+1/2 candidate needs sum(d) even (its coordinates are d + 1/2).

The decision between the two candidates is the sign of

    D = sum_i e_i - 2 + odd1 * (1 - 2 e_p) - odd2 * 2 e_r        (D < 0  <=>  D8 wins)

which must be exact.  ``nearest_e8`` evaluates it in fp64 on exact inputs and recomputes
it with exact rationals whenever the fp64 value is within 1e-9 of zero.
"""

from fractions import Fraction

import numpy as np

# Generator of 2E8 from App. E.  Row i gives X_i = sum_j GEN[i, j] c_j: the lattice point
# with coordinates c is GEN @ c (the lattice is the integer span of the columns).
GEN = np.array(
    [
        [1, 0, 0, 0, 0, 0, 0, 0],
        [1, 0, 2, 0, 0, 0, 0, 0],
        [1, 0, 0, 0, 2, 0, 0, 0],
        [1, 0, 0, 0, 0, 0, 2, 0],
        [1, 4, 2, 2, 2, 2, 2, 2],
        [1, 0, 0, 2, 0, 0, 0, 0],
        [1, 0, 0, 0, 0, 2, 0, 0],
        [1, 0, 0, 0, 0, 0, 0, 2],
    ],
    dtype=np.int64,
)


def _exact_inverse(m):
    """Gauss-Jordan inverse over the rationals (a textbook library step)."""
    n = m.shape[0]
    a = [[Fraction(int(m[i, j])) for j in range(n)] + [Fraction(int(i == j)) for j in range(n)]
         for i in range(n)]
    for col in range(n):
        piv = next(r for r in range(col, n) if a[r][col] != 0)
        a[col], a[piv] = a[piv], a[col]
        pv = a[col][col]
        a[col] = [v / pv for v in a[col]]
        for r in range(n):
            if r != col and a[r][col] != 0:
                fac = a[r][col]
                a[r] = [vr - fac * vc for vr, vc in zip(a[r], a[col])]
    return [row[n:] for row in a]


_GINV = _exact_inverse(GEN)
# det(GEN) = 2^8 and 4 * GEN^-1 is integral: keep the integer matrix and divide by 4.
GINV4 = np.array([[int(v * 4) for v in row] for row in _GINV], dtype=np.int64)
assert all((v * 4).denominator == 1 for row in _GINV for v in row)
assert np.array_equal(GINV4 @ GEN, 4 * np.eye(8, dtype=np.int64))


def in_2e8(P):
    """True where the integer 8-vector P lies in 2E8 (= 2 D8 u (2 D8 + 1)).

    2D8: all coordinates even with sum = 0 mod 4; 2(D8 + 1/2): all odd with sum = 0 mod 4.
    """
    P = np.asarray(P, dtype=np.int64)
    par = P & 1
    same = np.all(par == par[..., :1], axis=-1)
    return same & (P.sum(axis=-1) % 4 == 0)


def coordinates(P):
    """Coordinates v with GEN @ v = P for P in 2E8 (Alg. 1, second step)."""
    P = np.asarray(P, dtype=np.int64)
    v4 = P @ GINV4.T
    if np.any(v4 % 4):
        raise ValueError("point is not in 2E8")
    return v4 // 4


def _exact_gap(e_row, odd1, p, odd2, r):
    """The candidate gap D of the module docstring, in exact rationals."""
    e = [Fraction(float(v)) for v in e_row]
    D = sum(e) - 2
    if odd1:
        D += 1 - 2 * e[p]
    if odd2:
        D -= 2 * e[r]
    return D


def nearest_e8(y):
    """Q_E8(y) for exactly-representable float inputs (Alg. 5 with the readings above).

    y: float array of shape (..., 8) whose entries are exact binary fractions (fp32 values
    widened to fp64 are); every intermediate below is then exact except the candidate gap,
    whose sign is settled exactly.  (The distance to the nearest integer is taken as
    |y - rint(y)|, which is exact; y - floor(y) is not, for tiny negative y.)  Returns
    P = 2 Q_E8(y) as int64 of the same shape.
    """
    y = np.asarray(y, dtype=np.float64)
    shape = y.shape
    y = y.reshape(-1, 8)
    n = y.shape[0]
    rows = np.arange(n)

    d = np.floor(y)
    g = y > d + 0.5                        # round up (an exact half rounds down)
    e = np.abs(y - np.rint(y))             # distance to the nearest integer: exact
    s = np.where(g, 1, -1).astype(np.int64)
    di = d.astype(np.int64)

    x1 = di + g                            # nearest integer vector
    odd1 = (x1.sum(axis=1) & 1).astype(bool)
    p = np.argmax(e, axis=1)               # first maximum = lowest index
    x1[rows[odd1], p[odd1]] -= s[rows[odd1], p[odd1]]

    h2 = 2 * di + 1                        # 2 * (d + 1/2)
    odd2 = (di.sum(axis=1) & 1).astype(bool)
    r = np.argmin(e, axis=1)               # first minimum = lowest index
    h2[rows[odd2], r[odd2]] += 2 * s[rows[odd2], r[odd2]]

    e_p = e[rows, p]
    e_r = e[rows, r]
    gap = e.sum(axis=1) - 2.0 + odd1 * (1.0 - 2.0 * e_p) - odd2 * (2.0 * e_r)
    d8 = gap < 0
    for i in np.nonzero(np.abs(gap) < 1e-9)[0]:
        d8[i] = _exact_gap(e[i], odd1[i], p[i], odd2[i], r[i]) < 0

    P = np.where(d8[:, None], 2 * x1, h2)
    return P.reshape(shape)


def nearest_e8_rational(num, den):
    """Q_E8(num / den) for integer numerators and a positive integer denominator.

    Same algorithm and tie rules as ``nearest_e8`` but in exact integer arithmetic: all
    distances are kept multiplied by ``den``.  Used by the decoder (App. E), whose inputs are
    X / (2q) with X integral.  Returns P = 2 Q_E8(num / den) as int64.
    """
    num = np.asarray(num, dtype=np.int64)
    shape = num.shape
    num = num.reshape(-1, 8)
    den = int(den)
    n = num.shape[0]
    rows = np.arange(n)

    d = num // den                         # floor
    f = num - den * d                      # den * fractional part, in [0, den)
    e = np.minimum(f, den - f)             # den * distance to nearest integer
    g = 2 * f > den                        # strictly past the half
    s = np.where(g, 1, -1).astype(np.int64)

    x1 = d + g
    odd1 = (x1.sum(axis=1) & 1).astype(bool)
    p = np.argmax(e, axis=1)
    x1[rows[odd1], p[odd1]] -= s[rows[odd1], p[odd1]]

    h2 = 2 * d + 1
    odd2 = (d.sum(axis=1) & 1).astype(bool)
    r = np.argmin(e, axis=1)
    h2[rows[odd2], r[odd2]] += 2 * s[rows[odd2], r[odd2]]

    gap = e.sum(axis=1) - 2 * den + odd1 * (den - 2 * e[rows, p]) - odd2 * (2 * e[rows, r])
    d8 = gap < 0
    P = np.where(d8[:, None], 2 * x1, h2)
    return P.reshape(shape)


def nearest_e8_m_rational(num, den):
    """The NestQuantM oracle f (App. D) at num / den, in exact integer arithmetic.

    Alg. 5 with the parity of each candidate fixed at the first coordinate: the D8 candidate
    (nearest integer vector, halves down) moves its first coordinate to the other
    neighbouring integer when its sum is odd; the D8+1/2 candidate (d + 1/2) moves its first
    coordinate to the other neighbouring half-integer, towards the input, when sum d is odd.
    The closer candidate wins, a tie going to D8+1/2 as in ``nearest_e8``.  Distances are
    kept multiplied by den.  Returns 2 f(num / den) as int64.
    """
    num = np.asarray(num, dtype=np.int64)
    shape = num.shape
    num = num.reshape(-1, 8)
    den = int(den)

    d = num // den
    f = num - den * d
    e = np.minimum(f, den - f)             # den * distance to the nearest integer
    g = 2 * f > den
    s = np.where(g, 1, -1).astype(np.int64)

    x1 = d + g
    odd1 = (x1.sum(axis=1) & 1).astype(bool)
    x1[odd1, 0] -= s[odd1, 0]

    h2 = 2 * d + 1
    odd2 = (d.sum(axis=1) & 1).astype(bool)
    h2[odd2, 0] += 2 * s[odd2, 0]

    e0 = e[:, 0]
    gap = e.sum(axis=1) - 2 * den + odd1 * (den - 2 * e0) - odd2 * (2 * e0)
    d8 = gap < 0
    P = np.where(d8[:, None], 2 * x1, h2)
    return P.reshape(shape)
