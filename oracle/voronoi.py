"""Voronoi codes over 2E8 with nesting ratio q (Sec. 4.1, Alg. 1 and Alg. 2).

TEST INFRASTRUCTURE ONLY (see the package docstring).

The codebook is the set of points of the lattice inside q times its Voronoi region
(Sec. 4.1, definition of the Voronoi code); a point is sent as its coordinates mod q.

* Encode (Alg. 1): p = Q(x); v = G^-1 p; return v mod q.
* Decode (Alg. 2): p = G c; return p - q Q(p / q).

All points are in 2E8 units (P = 2 p, App. E), so with Lambda = 2E8 the decoder's
q Q_Lambda(P / q) equals q * 2 Q_E8(P / (2q)); ``decode`` evaluates it exactly with
integer arithmetic over the denominator 2q.

Overload (Sec. 4.1): the reconstruction equals Q(x) exactly when Q(x) lies in the shaping
region q V; otherwise the quantizer is in overload.  Because Alg. 5 breaks ties in a fixed
way, the literal test "decode(encode(P)) != P" is the definition used here.

NestQuantM (App. D) keeps the encoder and replaces the decoder's oracle by f (parity fixed at
the first coordinate); its shaping region is then {P : f(P / 2q) = 0} rather than q V, and
overload is again the literal test with that decoder.  ``decoder`` selects "full" (Alg. 2
with Alg. 5) or "m" (NestQuantM).
"""

import numpy as np

from .lattice import GEN, coordinates, nearest_e8_m_rational, nearest_e8_rational

DECODERS = ("full", "m")


def encode_point(P, q):
    """Alg. 1 after the nearest-point step: codes v mod q of the 2E8 point P, in [0, q)."""
    return np.mod(coordinates(P), int(q))


def decode(c, q, decoder="full"):
    """Alg. 2: the representative of the coset G c + q 2E8 chosen by the decoder (2E8 units)."""
    c = np.asarray(c, dtype=np.int64)
    X = c @ GEN.T                                    # X = G c for every 8-block
    if decoder == "full":
        return X - int(q) * nearest_e8_rational(X, 2 * int(q))
    if decoder == "m":
        return X - int(q) * nearest_e8_m_rational(X, 2 * int(q))
    raise ValueError(decoder)


def overloaded(P, q, decoder="full"):
    """True where the 2E8 point P is not reproduced by decode(encode(P))."""
    P = np.asarray(P, dtype=np.int64)
    return np.any(decode(encode_point(P, q), q, decoder) != P, axis=-1)
