"""Pins of the NestQuantM oracle f and its Voronoi-style code (App. D).

f is Alg. 5 with both parity fixes at the first coordinate.  What the paper and the
mathematics fix about it, and what these tests check:

* f(x) is a point of E8 (both candidates are lattice points);
* App. D's lemma: f(x + v) = f(x) + v for v in E8.  For v in D8 it holds for every x (the
  same roundings, parities and flip); for v in D8 + 1/2 the two candidates swap, so it holds
  whenever the candidates are not at equal distance;
* f equals the nearest point Q_E8 whenever neither candidate needs a parity fix;
* decoding with f is a bijection from the q^8 codes onto coset representatives (encode of
  the decoded point gives the code back), checked for every code at q = 2, 3, 4;
* App. D's derivation: decode_M(encode(P)) = P exactly when f(P / q) = 0 (2E8 units:
  f(P / 2q) = 0), whenever the code's coset shift is in D8;
* every decoded point lies in the box |P_0| <= 2q, |P_i| <= q (i > 0): the residual
  x - f(x) has coordinates within 1/2 of the rounding except the flipped first one, within
  1.  The GPU encoder uses this box to skip betas that surely overload.
"""

import itertools

import numpy as np
import pytest

from oracle import lattice, nestquant, voronoi


def _random_rational(rng, n, den, span):
    num = rng.integers(-span * den, span * den, size=(n, 8))
    return num, den


def _random_2e8(rng, n, span):
    coords = rng.integers(-span, span + 1, size=(n, 8))
    return coords @ lattice.GEN.T


def test_f_returns_e8_points():
    rng = np.random.default_rng(1)
    for den in (2, 7, 28, 1000003):
        num, _ = _random_rational(rng, 5000, den, 5)
        P = lattice.nearest_e8_m_rational(num, den)
        assert lattice.in_2e8(P).all()


def test_f_lemma_d8_shifts_exact_everywhere():
    """f(x + u) = f(x) + u for u in D8, for every x, ties included (halves, equal
    distances): x on a grid of step 1/4 makes exact halves and equal distances common."""
    rng = np.random.default_rng(2)
    den = 4
    num = rng.integers(-12, 13, size=(20000, 8))
    u = rng.integers(-3, 4, size=(20000, 8))
    u[:, 0] += u.sum(axis=1) & 1                      # even sum: u in D8
    base = lattice.nearest_e8_m_rational(num, den)
    shifted = lattice.nearest_e8_m_rational(num + den * u, den)
    assert np.array_equal(shifted, base + 2 * u)


def test_f_lemma_e8_shifts_off_ties():
    """f(x + v) = f(x) + v for v in E8 (here v = V / 2 with V in 2E8), on random x with a
    large odd denominator, where equal candidate distances do not occur."""
    rng = np.random.default_rng(3)
    den = 2 * 1000003                                 # even, so den * V / 2 is integral
    num, _ = _random_rational(rng, 20000, den, 4)
    V = _random_2e8(rng, 20000, 3)
    base = lattice.nearest_e8_m_rational(num, den)
    shifted = lattice.nearest_e8_m_rational(num + (den // 2) * V, den)
    assert np.array_equal(shifted, base + V)


def test_f_is_q_e8_without_parity_fixes():
    """Where round(x) (halves down) and floor(x) both have an even sum, no coordinate is
    flipped and f(x) = Q_E8(x)."""
    rng = np.random.default_rng(4)
    den = 1000003
    num, _ = _random_rational(rng, 40000, den, 4)
    d = num // den
    x1 = d + (2 * (num - den * d) > den)
    clean = ((x1.sum(axis=1) & 1) == 0) & ((d.sum(axis=1) & 1) == 0)
    assert clean.sum() > 5000
    f = lattice.nearest_e8_m_rational(num[clean], den)
    q = lattice.nearest_e8_rational(num[clean], den)
    assert np.array_equal(f, q)
    # and where a fix is needed the two oracles do differ sometimes (the variant is real)
    f_all = lattice.nearest_e8_m_rational(num, den)
    q_all = lattice.nearest_e8_rational(num, den)
    assert (f_all != q_all).any(axis=1).sum() > 100


@pytest.mark.parametrize("q", [2, 3, 4])
def test_decoder_m_is_a_bijection(q):
    codes = np.array(list(itertools.product(range(q), repeat=8)), dtype=np.int64)
    P = voronoi.decode(codes, q, "m")
    assert lattice.in_2e8(P).all()
    assert np.array_equal(voronoi.encode_point(P, q), codes)
    assert len({tuple(p) for p in P}) == q ** 8


@pytest.mark.parametrize("q", [2, 3, 4, 5])
def test_decoder_m_region_box(q):
    """Every point the NestQuantM decoder can return lies in |P_0| <= 2q, |P_i| <= q, and
    the box is tight (both bounds are reached)."""
    if q <= 4:
        codes = np.array(list(itertools.product(range(q), repeat=8)), dtype=np.int64)
    else:
        codes = np.random.default_rng(q).integers(0, q, size=(300000, 8))
    P = voronoi.decode(codes, q, "m")
    assert (np.abs(P[:, 0]) <= 2 * q).all()
    assert (np.abs(P[:, 1:]) <= q).all()
    assert (np.abs(P[:, 0]) == 2 * q).any() and (np.abs(P[:, 1:]) == q).any()


@pytest.mark.parametrize("q", [7, 14, 16])
def test_decoder_m_reproduces_exactly_its_region(q):
    """decode_M(encode(P)) = P exactly when f(P / 2q) = 0, for codes whose coset shift
    (G encode(P) - P) / 2q lies in D8 (App. D's derivation, exact in that case)."""
    rng = np.random.default_rng(10 + q)
    P = np.concatenate([_random_2e8(rng, 30000, 2 * q // 3), _random_2e8(rng, 30000, q // 3)])
    codes = voronoi.encode_point(P, q)
    X = codes @ lattice.GEN.T
    w2 = (X - P) // q                                  # 2 w, w = (X - P) / 2q in E8
    in_d8 = (w2 % 2 == 0).all(axis=1)
    assert in_d8.sum() > 10000
    back = voronoi.decode(codes[in_d8], q, "m")
    same = (back == P[in_d8]).all(axis=1)
    f_zero = (lattice.nearest_e8_m_rational(P[in_d8], 2 * q) == 0).all(axis=1)
    assert np.array_equal(same, f_zero)
    assert same.sum() > 100 and (~same).sum() > 100


def test_nestquantm_first_beta_uses_its_decoder():
    """With decoder "m", First-beta keeps the smallest t whose point the NestQuantM decoder
    reproduces, and every kept point (t < k) is reproduced exactly."""
    rng = np.random.default_rng(5)
    x = rng.standard_normal((64, 256)).astype(np.float32)
    q, k = 16, 4
    codes, t, r = nestquant.quantize_rows(x, q, k, decoder="m")
    c = nestquant.multipliers(r, k, nestquant.default_base(q, k))
    xb = x.reshape(-1, 8)
    cb = codes.reshape(-1, 8)
    tb = t.reshape(-1)
    mb = np.repeat(c, 32, axis=0)
    for i in range(0, xb.shape[0], 7):
        y = (xb[i] * mb[i, tb[i] - 1]).astype(np.float32).astype(np.float64)
        P = lattice.nearest_e8(y)
        assert np.array_equal(voronoi.encode_point(P, q), cb[i])
        if tb[i] < k:
            assert np.array_equal(voronoi.decode(cb[i], q, "m"), P)
        for s in range(1, tb[i]):
            ys = (xb[i] * mb[i, s - 1]).astype(np.float32).astype(np.float64)
            assert voronoi.overloaded(lattice.nearest_e8(ys), q, "m")
