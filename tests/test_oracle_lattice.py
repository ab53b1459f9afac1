"""Pins of the oracle's E8 primitives against what the paper and the mathematics fix.

* G is a basis of 2E8 (App. E): its columns lie in 2E8 and det G = 2^8 = covolume of 2E8,
  so they generate all of 2E8.
* Q_E8 is the nearest point of E8 (Sec. 3 eq. QLdef): brute force over every D8 and
  D8+1/2 point near the input, on random and on tie-heavy inputs.
* NSM of E8 = 0.0716821 (Sec. 3) by Monte Carlo.
* The integer (decoder) and float (encoder) forms of Alg. 5 agree on dyadic inputs.
* The update of Delta printed in Alg. 5 for the D8 parity fix returns points that are not
  nearest; the corrected update does not (the reading taken in the oracle).
"""

import itertools
from fractions import Fraction

import numpy as np
import pytest

from conftest import read_golden
from oracle import lattice, theory


def e8_roots():
    """The 240 minimal vectors of E8: +-e_i +- e_j and (+-1/2)^8 with an even number of minus signs."""
    roots = []
    for i, j in itertools.combinations(range(8), 2):
        for si, sj in itertools.product((1, -1), repeat=2):
            v = np.zeros(8)
            v[i], v[j] = si, sj
            roots.append(v)
    for signs in itertools.product((0.5, -0.5), repeat=8):
        if sum(s < 0 for s in signs) % 2 == 0:
            roots.append(np.array(signs))
    return np.array(roots)


def test_roots_count():
    R = e8_roots()
    assert R.shape == (240, 8)
    assert np.allclose((R * R).sum(1), 2.0)


def _det_exact(m):
    a = [[Fraction(int(v)) for v in row] for row in m]
    n, det = len(a), Fraction(1)
    for c in range(n):
        p = next((r for r in range(c, n) if a[r][c] != 0), None)
        if p is None:
            return 0
        if p != c:
            a[c], a[p] = a[p], a[c]
            det = -det
        det *= a[c][c]
        for r in range(c + 1, n):
            f = a[r][c] / a[c][c]
            a[r] = [x - f * y for x, y in zip(a[r], a[c])]
    return det


def test_generator_spans_2e8():
    G = lattice.GEN
    assert _det_exact(G) in (256, -256)
    assert np.all(lattice.in_2e8(G.T))                      # every column is in 2E8
    # 2E8 contains 2 * roots; all of them have integral coordinates in this basis
    R2 = (2 * e8_roots()).astype(np.int64)
    v = lattice.coordinates(R2)
    assert np.array_equal(v @ G.T, R2)


def test_generator_decomposition_identity():
    # App. E writes G as the sum of four simple matrices (all-ones first column, the 2's of
    # rows 1-3, the 2's on the diagonal-like positions of rows 4-7, and row 4's 2's).
    G = lattice.GEN
    M1 = np.zeros((8, 8), int); M1[:, 0] = 1
    M2 = np.zeros((8, 8), int); M2[1, 2] = M2[2, 4] = M2[3, 6] = 2
    M3 = np.zeros((8, 8), int); M3[4, 1] = M3[5, 3] = M3[6, 5] = M3[7, 7] = 2
    M4 = np.zeros((8, 8), int); M4[4, 1:] = 2
    assert np.array_equal(M1 + M2 + M3 + M4, G)


def brute_nearest(y):
    """All E8 points at minimal distance from y (exact rational distances)."""
    yi = np.round(y)
    offs = np.array(list(itertools.product((-1, 0, 1), repeat=8)))
    Z = yi[None, :] + offs
    Z = Z[(Z.sum(1) % 2) == 0]
    H = np.floor(y)[None, :] + 0.5 + offs
    H = H[(np.round((H - 0.5).sum(1)) % 2) == 0]
    C = np.concatenate([Z, H])
    d = ((C - y[None, :]) ** 2).sum(1)
    m = d.min()
    near = C[d <= m + 1e-9]
    yf = [Fraction(float(v)) for v in y]
    ex = [sum((Fraction(float(c)) - a) ** 2 for c, a in zip(row, yf)) for row in near]
    mex = min(ex)
    return np.array([row for row, v in zip(near, ex) if v == mex])


def adversarial_inputs(rng, n):
    out = []
    for _ in range(n):
        kind = rng.integers(0, 7)
        if kind == 0:     # exact halves and integers
            y = rng.integers(-6, 6, 8) + rng.choice([0.0, 0.5], 8)
        elif kind == 1:   # repeated distances: values sharing a fractional part
            fr = rng.choice([0.125, 0.25, 0.375, 0.625, 0.75], 8)
            y = rng.integers(-4, 4, 8) + fr
        elif kind == 2:   # D8 and D8+1/2 at equal distance: sum of e_i = 2 with even sums
            y = np.full(8, 0.25) + 2 * rng.integers(-2, 2, 8)
        elif kind == 3:   # quarter grid
            y = rng.integers(-16, 16, 8) / 4.0
        elif kind == 4:   # tiny values near 0 with a few halves
            y = rng.standard_normal(8) * 1e-6
            y[rng.integers(0, 8)] = 0.5
        elif kind == 5:   # eighth grid
            y = rng.integers(-40, 40, 8) / 8.0
        else:             # tiny entries of both signs next to exact zeros and halves
            y = rng.choice([0.0, 0.5, -0.5, 1.0], 8)
            k = rng.integers(1, 4)
            y[:k] = rng.choice([-1.0, 1.0], k) * 10.0 ** rng.uniform(-30, -8, k)
        out.append(y.astype(np.float32).astype(np.float64))
    return np.array(out)


def test_nearest_matches_brute_force(rng):
    ys = np.concatenate([
        (rng.standard_normal((600, 8)) * 3).astype(np.float32).astype(np.float64),
        (rng.uniform(-20, 20, (200, 8))).astype(np.float32).astype(np.float64),
        adversarial_inputs(rng, 600),
    ])
    P = lattice.nearest_e8(ys)
    assert np.all(lattice.in_2e8(P))
    ties = 0
    for i in range(len(ys)):
        best = brute_nearest(ys[i])
        got = P[i] / 2.0
        assert any(np.array_equal(got, b) for b in best), (ys[i], got, best)
        if len(best) == 1:
            assert np.array_equal(got, best[0])
        else:
            ties += 1
    assert ties > 50          # the adversarial set does exercise ties


def test_tie_rules():
    # exact half rounds down, argmin/argmax take the lowest index, D = 0 goes to D8+1/2
    y = np.full(8, 0.25)                     # D8 point 0 and D8+1/2 point 1/2 at equal distance
    assert np.array_equal(lattice.nearest_e8(y), np.ones(8, np.int64))
    y = np.array([0.5, 0, 0, 0, 0, 0, 0, 0.0])
    # the exact half rounds down: D8 point 0 at distance 1/4 (the unique nearest point)
    assert np.array_equal(lattice.nearest_e8(y), np.zeros(8, np.int64))


def test_nsm_monte_carlo():
    (nsm_row,) = [r for r in read_golden("constants.txt") if r[0] == "nsm_e8"]
    rng = np.random.default_rng(7)
    y = rng.uniform(0.0, 2.0, (400000, 8)).astype(np.float32).astype(np.float64)
    P = lattice.nearest_e8(y)
    err = ((y - P / 2.0) ** 2).sum(1) / 8.0
    est, se = err.mean(), err.std() / np.sqrt(len(err))
    assert abs(est - float(nsm_row[1])) < 5 * se + 1e-7
    assert abs(theory.NSM_E8 - float(nsm_row[1])) < 1e-7


def test_rational_form_matches_float_form(rng):
    for q in (2, 4, 8, 16):
        X = rng.integers(-200, 200, (5000, 8))
        a = lattice.nearest_e8_rational(X, 2 * q)
        b = lattice.nearest_e8((X / (2.0 * q)))
        assert np.array_equal(a, b)


def test_rational_form_brute_force(rng):
    for q in (3, 7, 14):
        X = rng.integers(-6 * q, 6 * q, (150, 8))
        P = lattice.nearest_e8_rational(X, 2 * q)
        for i in range(len(X)):
            y = [Fraction(int(v), 2 * q) for v in X[i]]
            d = lambda z: sum((Fraction(float(c)) - a) ** 2 for c, a in zip(z, y))  # noqa: E731
            got = d(P[i] / 2.0)
            # compare with the brute-force minimum on the float image (exact enough to
            # locate candidates), then exactly
            best = brute_nearest(np.array([float(v) for v in y]))
            assert got == min(d(b) for b in best)


def test_equivariance_under_d8_shifts(rng):
    y = (rng.standard_normal((3000, 8)) * 2).astype(np.float32).astype(np.float64)
    v = rng.integers(-3, 3, (3000, 8))
    v[:, 0] += v.sum(1) % 2                     # make the sum even: v in D8
    assert np.array_equal(lattice.nearest_e8(y + v), lattice.nearest_e8(y) + 2 * v)


def _printed_alg5(y):
    """Alg. 5 with Delta updated as printed for the D8 parity fix (+2 dist - 1)."""
    d = np.floor(y)
    x2 = d + 0.5
    g = y > x2
    s = 2 * g - 1
    x1 = d + g
    dist = (y - x2) * s
    delta = dist.sum()
    if int(x1.sum()) % 2:
        pos = int(np.argmin(dist))
        x1[pos] -= s[pos]
        delta += 2 * dist[pos] - 1
    if int(d.sum()) % 2:
        pos = int(np.argmax(dist))
        x2[pos] += s[pos]
        delta += 1 - 2 * dist[pos]
    return x1 if delta > 2 else x2


def test_printed_delta_update_is_an_erratum():
    rng = np.random.default_rng(3)
    ys = (rng.standard_normal((1500, 8)) * 2).astype(np.float32).astype(np.float64)
    ours = lattice.nearest_e8(ys) / 2.0
    wrong = 0
    for i, y in enumerate(ys):
        p = _printed_alg5(y.copy())
        dp = ((p - y) ** 2).sum()
        do = ((ours[i] - y) ** 2).sum()
        assert do <= dp + 1e-12
        wrong += dp > do + 1e-12
    assert wrong > 100


def test_r_star():
    (row,) = [r for r in read_golden("constants.txt") if r[0] == "r_star"]
    assert abs(theory.r_star() - float(row[1])) < 5e-4
