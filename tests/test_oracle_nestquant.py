"""Pins of the oracle's row quantizer, decoder and coded product.

* App. F, Table rmse-beta: pooled RMSE of First-beta and Opt-beta on iid N(0,1) 8-vectors
  at q = 16 with k betas uniform on [0, 10] / q (golden file, +-0.0006).
* Rate (Sec. 3, "union of Voronoi codes"): log2 q + log2(k)/8 against the printed
  "Bits (no zstd)" column and the 4.25 bits of the GEMV table.
* Row scale: the fp32 number nearest the exact RMS, checked by exact rational arithmetic,
  plus special cases (constant rows, zero rows, power-of-two scaling invariance).
* First-beta: the chosen beta is the smallest one that does not overload, else the largest.
* A lattice point inside the shaping region is reproduced exactly.
* Coded product: equals Alg. 4 row by row, and the textbook product of the decoded
  matrices; on Gaussian data its error lies above the Gamma(R) lower bound (Sec. 2.1).
"""

import math
from fractions import Fraction

import numpy as np
import pytest

from conftest import read_golden
from oracle import layout, lattice, nestquant, theory, voronoi
from test_oracle_voronoi import root_bound


def test_rmse_beta_table():
    rng = np.random.default_rng(2024)
    v = rng.standard_normal((60000, 8)).astype(np.float32)
    q = 16
    for k_s, opt_s, first_s in read_golden("rmse_beta_table.txt"):
        k = int(k_s)
        betas = 10.0 * np.arange(1, k + 1) / k / q
        mult = np.tile((1.0 / betas).astype(np.float32), (len(v), 1))
        res = {}
        for strat in ("opt", "first"):
            codes, t, _, _ = nestquant.quantize_blocks(v, mult, q, strat, v.astype(np.float64), betas)
            rec = betas[t - 1][:, None] * voronoi.decode(codes, q) / 2.0
            res[strat] = math.sqrt(((rec - v) ** 2).mean())
        assert abs(res["opt"] - float(opt_s)) < 6e-4, (k, res)
        assert abs(res["first"] - float(first_s)) < 6e-4, (k, res)
        assert res["opt"] <= res["first"] + 1e-12


def test_rate_bits():
    for q, k, bits in read_golden("rate_bits.txt"):
        assert round(theory.rate_bits(int(q), int(k)), 2) == float(bits)


def _exact_rms(row):
    S = sum(Fraction(float(v)) ** 2 for v in row)
    return S / len(row)


def _is_nearest_f32(r32, t):
    """r32 is the fp32 number nearest to sqrt(t) (ties to even)."""
    r = Fraction(float(r32))
    lo = Fraction(float(np.nextafter(np.float32(r32), np.float32(-np.inf))))
    hi = Fraction(float(np.nextafter(np.float32(r32), np.float32(np.inf))))
    m_lo, m_hi = (lo + r) / 2, (r + hi) / 2
    return (r32 == 0 or m_lo * m_lo <= t) and t <= m_hi * m_hi


def test_row_scale_exact(rng):
    for dtype in ("f32", "bf16", "f16"):
        from workloads import random_rows
        _, x = random_rows(11, 200, 64, dtype=dtype, scale=3.0)
        r = nestquant.row_scale(x)
        for i in range(x.shape[0]):
            assert _is_nearest_f32(r[i], _exact_rms(x[i]))


def test_row_scale_special_rows():
    # constant rows: the RMS is |a| exactly
    for a in (1.0, 0.1, 3.0e-20, 7.5e30, 1.401298464324817e-45):
        x = np.full((1, 16), a, dtype=np.float32)
        assert nestquant.row_scale(x)[0] == np.float32(a)
    x = np.zeros((2, 8), np.float32)
    x[1, 3] = -2.0
    r = nestquant.row_scale(x)
    assert r[0] == 0 and r[1] == np.float32(2.0 / math.sqrt(8))
    # (1, 1 + d) with d = 2^-23: RMS = 1 + d/2 + d^2/8 + O(d^3), just above the midpoint
    # 1 + d/2 between the fp32 numbers 1 and 1 + d, so it rounds up to 1 + d.  The fp64
    # estimate lies within 1e-9 of the midpoint, so this exercises the exact path.
    d = 2.0 ** -23
    x = np.array([[1.0, 1.0 + d]], np.float32)
    assert nestquant.row_scale(x)[0] == np.float32(1.0 + d)
    # (1, 1 - d/2): RMS = 1 - d/4 + d^2/64 + O(d^3), just above the midpoint 1 - d/4
    # between 1 - d/2 and 1, so it rounds up to 1.
    x = np.array([[1.0, 1.0 - d / 2]], np.float32)
    assert nestquant.row_scale(x)[0] == np.float32(1.0)


def test_row_scale_fast_path_agrees_with_exact(rng):
    from workloads import random_rows
    _, x = random_rows(13, 300, 40, dtype="f32", dist="t4")
    r = nestquant.row_scale(x)
    for i in range(x.shape[0]):
        assert r[i] == nestquant._exact_rms_f32(x[i])


def test_scaling_invariance(rng):
    from workloads import random_rows
    _, x = random_rows(5, 40, 128, dtype="bf16")
    c0, t0, r0 = nestquant.quantize_rows(x, 14, 4)
    for e in (-20, -3, 5, 17):
        c1, t1, r1 = nestquant.quantize_rows(x * np.float32(2.0 ** e), 14, 4)
        assert np.array_equal(c0, c1) and np.array_equal(t0, t1)
        assert np.array_equal(r1, r0 * np.float32(2.0 ** e))


def test_zero_rows():
    x = np.zeros((3, 32), np.float32)
    x[1] = np.arange(32)
    c, t, r = nestquant.quantize_rows(x, 14, 4)
    assert r[0] == 0 and r[2] == 0 and r[1] > 0
    assert not c[0].any() and not c[2].any()
    assert np.all(t[0] == 1) and np.all(t[2] == 1)
    assert not nestquant.decode_rows(c, t, r, 14, nestquant.default_base(14, 4))[0].any()


def test_first_beta_rule(rng):
    from workloads import random_rows
    _, x = random_rows(9, 64, 256, dtype="f32", dist="t4")
    q, k = 7, 4
    base = nestquant.default_base(q, k)
    r = nestquant.row_scale(x)
    mult = nestquant.multipliers(r, k, base)
    xb = x.reshape(-1, 8)
    mb = np.repeat(mult, 32, axis=0)
    codes, t, over, P = nestquant.quantize_blocks(xb, mb, q, "first")
    for i in range(len(t)):
        ok = np.nonzero(~over[i])[0]
        assert t[i] == (ok[0] + 1 if len(ok) else k)
    assert (t == k).sum() > 0 and (t == 1).sum() > 0
    # codes are those of the chosen beta's point
    rows = np.arange(len(t))
    assert np.array_equal(voronoi.encode_point(P[rows, t - 1], q), codes)
    assert np.all((codes >= 0) & (codes < q))


def test_beta_multiples_scaled_grid_is_the_same_code():
    """beta_t = m_t * base with m_t = 4 t and base / 4 is the uniform grid t * base exactly
    (a power-of-two rescaling), so the codes, indices and scales are identical."""
    from workloads import random_rows
    _, x = random_rows(14, 24, 256, dtype="bf16", dist="t4")
    base = nestquant.default_base(14, 4)
    c0, t0, r0 = nestquant.quantize_rows(x, 14, 4)
    c1, t1, r1 = nestquant.quantize_rows(x, 14, 4, base / 4, mult=(4, 8, 12, 16))
    assert np.array_equal(c0, c1) and np.array_equal(t0, t1) and np.array_equal(r0, r1)
    d0 = nestquant.decode_rows(c0, t0, r0, 14, base)
    d1 = nestquant.decode_rows(c1, t1, r1, 14, base / 4, mult=(4, 8, 12, 16))
    assert np.array_equal(d0, d1)


@pytest.mark.parametrize("mult,q", [((6, 8, 10, 15), 16), ((3, 5, 9), 14), ((7,), 7)])
def test_first_beta_rule_with_beta_multiples(mult, q):
    """With an arbitrary increasing beta set, First-beta keeps the first beta whose point
    survives decode(encode(.)), re-derived here block by block from the definition."""
    from workloads import random_rows
    _, x = random_rows(15 + q, 16, 256, dtype="f32", dist="t4")
    k, base = len(mult), 1.0 / (2 * q)
    codes, t, r = nestquant.quantize_rows(x, q, k, base, mult=mult)
    xb, cb, tb = x.reshape(-1, 8), codes.reshape(-1, 8), t.reshape(-1)
    rb = np.repeat(r, 32)
    for i in range(0, xb.shape[0], 5):
        pts = []
        for m in mult:
            c = np.float32(1.0 / (np.float64(rb[i]) * (np.float64(m) * base)))
            pts.append(lattice.nearest_e8((xb[i] * c).astype(np.float32).astype(np.float64)))
        ok = [not voronoi.overloaded(P, q) for P in pts]
        want = ok.index(True) + 1 if any(ok) else k
        assert tb[i] == want
        assert np.array_equal(voronoi.encode_point(pts[want - 1], q), cb[i])


def test_coded_product_with_beta_multiples():
    from workloads import random_rows
    _, A = random_rows(23, 5, 64, dtype="f32")
    _, W = random_rows(24, 4, 64, dtype="bf16", scale=0.02)
    ma, mw, q = (6, 8, 10, 15), (2, 3, 5, 11), 14
    base = 1.0 / (2 * q)
    ca, ta, ra = nestquant.quantize_rows(A, q, 4, base, mult=ma)
    cw, tw, rw = nestquant.quantize_rows(W, q, 4, base, mult=mw)
    C = nestquant.coded_matmul(ca, ta, ra, q, base, cw, tw, rw, q, base, mult_a=ma, mult_w=mw)
    for i in range(5):
        for j in range(4):
            ref = nestquant.dot_coded(ca[i], ta[i], ra[i], q, base, cw[j], tw[j], rw[j], q,
                                      base, ma, mw)
            assert C[i, j] == pytest.approx(ref, rel=1e-13, abs=1e-300)
    Ahat = nestquant.decode_rows(ca, ta, ra, q, base, mult=ma)
    What = nestquant.decode_rows(cw, tw, rw, q, base, mult=mw)
    assert np.allclose(C, Ahat @ What.T, rtol=1e-12, atol=0)


def test_lattice_points_reproduced(rng):
    q = 14
    # E8 points well inside q V: decode(encode) reproduces them exactly
    y = rng.standard_normal((5000, 8)) * 2
    P = lattice.nearest_e8(y.astype(np.float32).astype(np.float64))
    keep = root_bound(P) < 2 * q
    xb = (P[keep] / 2.0).astype(np.float32)
    codes, t, _, _ = nestquant.quantize_blocks(xb, np.ones((len(xb), 1), np.float32), q)
    assert np.array_equal(voronoi.decode(codes, q), P[keep])
    assert np.all(t == 1)


def test_coded_product_matches_alg4_and_decoded_product():
    from workloads import random_rows
    _, A = random_rows(21, 6, 64, dtype="f32")
    _, W = random_rows(22, 5, 64, dtype="bf16", scale=0.02)
    qa, qw, k = 14, 7, 4
    ba, bw = nestquant.default_base(qa, k), nestquant.default_base(qw, k)
    ca, ta, ra = nestquant.quantize_rows(A, qa, k)
    cw, tw, rw = nestquant.quantize_rows(W, qw, k)
    C = nestquant.coded_matmul(ca, ta, ra, qa, ba, cw, tw, rw, qw, bw)
    for i in range(6):
        for j in range(5):
            ref = nestquant.dot_coded(ca[i], ta[i], ra[i], qa, ba, cw[j], tw[j], rw[j], qw, bw)
            assert C[i, j] == pytest.approx(ref, rel=1e-13, abs=1e-300)
    Ahat = nestquant.decode_rows(ca, ta, ra, qa, ba)
    What = nestquant.decode_rows(cw, tw, rw, qw, bw)
    assert np.allclose(C, Ahat @ What.T, rtol=1e-12, atol=0)


def test_error_above_information_bound():
    from workloads import operand
    _, A, _ = operand(1, "A")
    _, W, _ = operand(1, "W")
    q, k = 14, 4
    base = nestquant.default_base(q, k)
    ca, ta, ra = nestquant.quantize_rows(A, q, k)
    cw, tw, rw = nestquant.quantize_rows(W, q, k)
    C = nestquant.coded_matmul(ca, ta, ra, q, base, cw, tw, rw, q, base)
    ref = A.astype(np.float64) @ W.astype(np.float64).T
    rel = np.linalg.norm(C - ref) / np.linalg.norm(ref)
    floor = math.sqrt(theory.gamma(theory.rate_bits(q, k)))
    assert floor < rel < 2 * floor


def test_layout_roundtrip(rng):
    c = rng.integers(0, 16, (7, 37, 8))
    w = layout.pack_codes(c)
    assert np.array_equal(layout.unpack_codes(w), c)
    assert layout.pack_codes(np.arange(8)[None, None, :])[0, 0] == 0x76543210
    t = rng.integers(1, 5, (7, 37))
    b = layout.pack_beta(t)
    assert b.shape == (7, 3)
    assert np.array_equal(layout.unpack_beta(b, 37), t)
    assert layout.pack_beta(np.array([[2, 1, 4]]))[0, 0] == (1 | (0 << 2) | (3 << 4))
