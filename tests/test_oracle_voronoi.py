"""Pins of the oracle's Voronoi code (Sec. 4.1, Alg. 1 and Alg. 2) against its definition.

* The codebook has q^8 points, one per coset of q 2E8 (Sec. 4.1): decode is injective on
  Z_q^8, and encode(decode(c)) = c, for every code at q = 2, 3, 4 and for random codes at
  q = 7, 14, 16.
* Decoded points lie in q V (the closed Voronoi cell of q 2E8), checked against the 240
  roots, and in the coset G c + q 2E8.
* Overload (Sec. 4.1): a point strictly inside q V is reproduced, one strictly outside
  is not.
"""

import itertools

import numpy as np
import pytest

from oracle import lattice, voronoi
from test_oracle_lattice import e8_roots

ROOTS = e8_roots()


def root_bound(P):
    """max over the 240 roots lambda of <P, lambda> (P in 2E8 units)."""
    return (np.asarray(P, np.float64) @ ROOTS.T).max(axis=-1)


@pytest.mark.parametrize("q", [2, 3, 4])
def test_bijection_all_codes(q):
    c = np.array(list(itertools.product(range(q), repeat=8)), dtype=np.int64)
    X2 = voronoi.decode(c, q)
    assert np.all(lattice.in_2e8(X2))
    assert len(np.unique(X2, axis=0)) == q ** 8
    assert np.array_equal(voronoi.encode_point(X2, q), c)
    assert np.all(root_bound(X2) <= 2 * q + 1e-9)
    assert np.all(np.abs(X2) <= 2 * q)


@pytest.mark.parametrize("q", [5, 7, 14, 16])
def test_roundtrip_random_codes(q, rng):
    c = rng.integers(0, q, (100000, 8))
    X2 = voronoi.decode(c, q)
    assert np.array_equal(voronoi.encode_point(X2, q), c)
    assert np.all(root_bound(X2) <= 2 * q + 1e-9)
    assert np.all(np.abs(X2) <= 2 * q)
    # same coset as G c
    diff = (c @ lattice.GEN.T) - X2
    assert np.all(diff % q == 0)
    assert np.all(lattice.in_2e8(diff // q))


@pytest.mark.parametrize("q", [3, 7, 14, 16])
def test_overload_criterion(q, rng):
    y = (rng.standard_normal((40000, 8)) * q * rng.uniform(0.1, 0.6, (40000, 1)))
    P = lattice.nearest_e8(y.astype(np.float32).astype(np.float64))
    M = root_bound(P)
    over = voronoi.overloaded(P, q)
    inside, outside = M < 2 * q - 1e-9, M > 2 * q + 1e-9
    assert inside.sum() > 1000 and outside.sum() > 1000
    assert not over[inside].any()
    assert over[outside].all()
    # on the boundary M = 2q both outcomes occur (tie-dependent)
    edge = ~inside & ~outside
    assert edge.sum() > 0
