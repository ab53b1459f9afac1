"""NestQuant row quantizer, decoder, dot product and coded matrix product.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Paper passages followed:

* Sec. 4.2, Alg. 3 (NestQuant): normalize a row of length n by s = ||A||_2 and sqrt(n);
  split it into n/8 blocks; code each block with the Voronoi code at one of k scaling
  coefficients beta_1 < ... < beta_k and keep the index of the one used.
* App. F, "First-beta": use the smallest beta that does not overload.  "Opt-beta" (the
  literal loop of Alg. 3): try every beta and keep the one with the smallest squared error
  (the first one on an exact tie, since Alg. 3 replaces only on a strict improvement); the
  error is ||beta_t X2_t / 2 - x / r||^2 in fp64, squares added in coordinate order.
* Sec. 3 "Overload avoidance via union of Voronoi codes": the codebook is the union of
  the k scaled Voronoi codes; the rate is log2(q) + log2(k)/8 bits per entry.
* Sec. 4.2, Alg. 4 (Dot product): sum over blocks of <p1, p2> beta_{B1} beta_{B2}.
* App. D (NestQuantM): the same encoder with overload judged by, and reconstruction made
  with, the NestQuantM decoder (``decoder="m"`` throughout).

Readings where the paper is silent:

* Row scale.  r = s / sqrt(n) = sqrt(sum_j x_j^2 / n) (the RMS), stored as the fp32 number
  nearest to the exact value (ties to even); a zero row has r = 0 and is coded as all-zero
  codes with beta index 1.
* Beta grid.  beta_t = t * base, t = 1..k, with base = 10 / (k q): App. F's table takes the
  k betas uniform on [0, 10], in the paper's "/q" units (App. G).  A set chosen by the
  dynamic program of App. F (from the grid (1/2) {1, ..., 50} / q) is given as integer
  multiples: beta_t = mult_t * base with mult_1 < ... < mult_k (``mult``; None = 1..k).
* Lattice input.  The multiplier for beta_t is c_t = fl32(1 / fl64(r * fl64(t * base)))
  (fp64 product, fp64 division, one rounding to fp32) and the block sent to the E8
  quantizer is y = fl32(x * c_t), computed with one fp32 multiply per entry.
* All betas overload: keep the largest (t = k), as Alg. 3 would keep some beta.
* Alg. 4 leaves out the normalization; the product is multiplied back by r1 * r2.
"""

from fractions import Fraction

import numpy as np

from .lattice import nearest_e8
from .voronoi import decode, encode_point


def default_base(q, k):
    """beta_t = t * base with the k betas uniform on [0, 10] / q (App. F table, App. G)."""
    return 10.0 / (k * q)


# ----------------------------------------------------------------------------------------
# Row scale (Alg. 3, the normalization coefficient)
# ----------------------------------------------------------------------------------------

def _f32_neighbours(v):
    v = np.float32(v)
    return np.nextafter(v, np.float32(-np.inf)), np.nextafter(v, np.float32(np.inf))


def _exact_rms_f32(row32):
    """RN_even_fp32(sqrt(sum x^2 / n)) with exact rational arithmetic."""
    n = row32.shape[0]
    S = sum(Fraction(float(v)) ** 2 for v in row32)
    if S == 0:
        return np.float32(0.0)
    t = S / n
    v = np.float32(np.sqrt(float(t)))

    def mid(a, b):
        return (Fraction(float(a)) + Fraction(float(b))) / 2

    while True:
        lo, hi = _f32_neighbours(v)
        m_hi, m_lo = mid(v, hi), mid(lo, v)
        if t > m_hi * m_hi:
            v = hi
        elif v > 0 and t < m_lo * m_lo:
            v = lo
        else:
            break
    even = (v.view(np.uint32) & 1) == 0
    lo, hi = _f32_neighbours(v)
    if t == mid(v, hi) ** 2 and not even:
        v = hi
    elif v > 0 and t == mid(lo, v) ** 2 and not even:
        v = lo
    return np.float32(v)


def row_scale(x32):
    """r_i = the fp32 number nearest to sqrt(sum_j x_ij^2 / n), per row.

    Fast path: fp64 sums, accepted only when the fp64 RMS is farther than 1e-9 (relative)
    from every fp32 rounding boundary; the fp64 value is far more accurate than that, so
    the rounding is then certain.  Other rows are recomputed exactly.
    """
    x32 = np.asarray(x32, dtype=np.float32)
    rows, n = x32.shape
    x64 = x32.astype(np.float64)
    r64 = np.sqrt(np.einsum("ij,ij->i", x64, x64) / n)
    r32 = r64.astype(np.float32)
    lo = np.nextafter(r32, np.float32(-np.inf)).astype(np.float64)
    hi = np.nextafter(r32, np.float32(np.inf)).astype(np.float64)
    c = r32.astype(np.float64)
    dist = np.minimum(np.abs(r64 - (c + lo) / 2), np.abs(r64 - (c + hi) / 2))
    unsure = ~(dist > 1e-9 * r64) | (r64 == 0) | ~np.isfinite(r64)
    for i in np.nonzero(unsure)[0]:
        r32[i] = _exact_rms_f32(x32[i])
    return r32


def beta_mults(k, mult=None):
    """The integer multiples m_t of base, t = 1..k (beta_t = m_t * base): 1..k by default."""
    if mult is None:
        return np.arange(1, k + 1, dtype=np.int64)
    m = np.asarray(mult, dtype=np.int64)[:k]
    if m.shape[0] != k or m[0] < 1 or (np.diff(m) <= 0).any():
        raise ValueError("mult must hold k strictly increasing positive integers")
    return m


def betas(k, base, mult=None):
    """beta_t = fl64(m_t * base), t = 1..k."""
    return beta_mults(k, mult).astype(np.float64) * np.float64(base)


def multipliers(r32, k, base, mult=None):
    """c_t = fl32(1 / fl64(r * fl64(m_t * base))) for t = 1..k; shape (rows, k).  Rows with
    r = 0 get 0 (they are coded as zeros and never multiplied)."""
    r64 = np.asarray(r32, dtype=np.float32).astype(np.float64)
    out = np.zeros((r64.shape[0], k), dtype=np.float32)
    nz = r64 != 0
    b = betas(k, base, mult)
    for t in range(1, k + 1):
        out[nz, t - 1] = (1.0 / (r64[nz] * b[t - 1])).astype(np.float32)
    return out


# ----------------------------------------------------------------------------------------
# Block quantizer: one 8-vector at k scales (Alg. 3 inner loop, App. F strategies)
# ----------------------------------------------------------------------------------------

def opt_errors(X2, v64, betas):
    """Opt-beta's reconstruction errors ||beta_t X2_t / 2 - v||^2 for every block and beta,
    (nb, k), in fp64 with the eight squares added left to right (a fixed order, so that the
    comparison between betas is reproducible)."""
    b = np.asarray(betas, dtype=np.float64)
    err = np.zeros(X2.shape[:2], dtype=np.float64)
    for l in range(8):
        d = b[None, :] * X2[:, :, l] / 2.0 - v64[:, None, l]
        err = err + d * d
    return err


def quantize_blocks(xb32, mult32, q, strategy="first", v64=None, betas=None, decoder="full"):
    """Quantize 8-blocks with the union of k scaled Voronoi codes.

    xb32:   (nb, 8) fp32 blocks.
    mult32: (nb, k) fp32 multipliers c_t (y_t = fl32(x * c_t) is the E8 input for beta_t).
    strategy: "first" (First-beta) or "opt" (Opt-beta; needs v64, the normalized blocks in
            fp64, and betas, the k beta values, to measure the error ||beta_t p - v||^2).
    Returns (codes (nb, 8) int64 in [0, q), t (nb,) int64 in [1, k], overload (nb, k) bool,
    P (nb, k, 8) the 2E8 points Q_E8(y_t)).
    """
    xb32 = np.asarray(xb32, dtype=np.float32)
    nb = xb32.shape[0]
    k = mult32.shape[1]
    P = np.empty((nb, k, 8), dtype=np.int64)
    codes = np.empty((nb, k, 8), dtype=np.int64)
    X2 = np.empty((nb, k, 8), dtype=np.int64)
    for t in range(k):
        y = (xb32 * mult32[:, t:t + 1]).astype(np.float32)   # one fp32 multiply per entry
        P[:, t] = nearest_e8(y.astype(np.float64))
        codes[:, t] = encode_point(P[:, t], q)
        X2[:, t] = decode(codes[:, t], q, decoder)
    over = np.any(X2 != P, axis=2)

    if strategy == "first":
        ok = ~over
        t_sel = np.where(ok.any(axis=1), np.argmax(ok, axis=1), k - 1)
    elif strategy == "opt":
        err = opt_errors(X2, v64, betas)
        t_sel = np.argmin(err, axis=1)                        # first minimum
    else:
        raise ValueError(strategy)
    rows = np.arange(nb)
    return codes[rows, t_sel], t_sel + 1, over, P


def quantize_rows(x, q, k, base=None, strategy="first", decoder="full", mult=None):
    """Alg. 3 on every row of x (rows, n), n a multiple of 8; x must be fp32-representable.
    beta_t = mult_t * base (mult None: t * base).

    Returns (codes (rows, n/8, 8) int64, t (rows, n/8) int64 in [1, k], r (rows,) fp32).
    """
    if base is None:
        base = default_base(q, k)
    x32 = np.asarray(x, dtype=np.float32)
    if not np.array_equal(x32.astype(np.float64), np.asarray(x, dtype=np.float64)):
        raise ValueError("input is not exactly representable in fp32")
    rows, n = x32.shape
    if n % 8:
        raise ValueError("row length must be a multiple of 8")
    nb = n // 8
    r = row_scale(x32)
    c = multipliers(r, k, base, mult)
    codes = np.zeros((rows, nb, 8), dtype=np.int64)
    t = np.ones((rows, nb), dtype=np.int64)
    nz = r != 0
    if nz.any():
        xb = x32[nz].reshape(-1, 8)
        mb = np.repeat(c[nz], nb, axis=0)
        v64 = bts = None
        if strategy == "opt":
            v64 = (x32[nz].astype(np.float64) / r[nz].astype(np.float64)[:, None]).reshape(-1, 8)
            bts = betas(k, base, mult)
        cb, tb, _, _ = quantize_blocks(xb, mb, q, strategy, v64, bts, decoder)
        codes[nz] = cb.reshape(-1, nb, 8)
        t[nz] = tb.reshape(-1, nb)
    return codes, t, r


# ----------------------------------------------------------------------------------------
# Decoding, dot product (Alg. 4) and the coded matrix product
# ----------------------------------------------------------------------------------------

def decoded_points(codes, q, decoder="full"):
    """Decoded lattice points in 2E8 units, X2 = 2 p (Alg. 2), same shape as codes."""
    return decode(codes, q, decoder)


def _mult_of(t, mult):
    """m_t for an array of beta indices t (1-based): t itself, or the table mult."""
    t = np.asarray(t, dtype=np.int64)
    if mult is None:
        return t
    return beta_mults(len(mult), mult)[t - 1]


def decode_rows(codes, t, r, q, base, decoder="full", mult=None):
    """Reconstruction x_hat = r * beta_t * p = r * base * m_t * X2 / 2 in fp64; (rows, n)."""
    X2 = decode(codes, q, decoder).astype(np.float64)       # (rows, nb, 8)
    scale = (np.asarray(r, np.float32).astype(np.float64)[:, None] * float(base)
             * _mult_of(t, mult).astype(np.float64) / 2.0)
    return (X2 * scale[:, :, None]).reshape(codes.shape[0], -1)


def dot_coded(c1, t1, r1, q1, base1, c2, t2, r2, q2, base2, mult1=None, mult2=None):
    """Alg. 4 for two coded vectors (blocks (nb, 8)): sum_j <p1_j, p2_j> beta1_j beta2_j,
    times the row scales r1 * r2 that Alg. 4 leaves out.  Plain loop, exact rationals
    (beta = base * m_t taken as exact rationals, not as the rounded fp64 betas)."""
    p1 = decode(np.asarray(c1), q1)
    p2 = decode(np.asarray(c2), q2)
    m1 = _mult_of(t1, mult1)
    m2 = _mult_of(t2, mult2)
    ans = Fraction(0)
    for j in range(p1.shape[0]):
        ip = Fraction(int(np.dot(p1[j], p2[j])), 4)           # <X2_1, X2_2> / 4 = <p1, p2>
        ans += ip * Fraction(base1) * int(m1[j]) * Fraction(base2) * int(m2[j])
    return float(ans * Fraction(float(r1)) * Fraction(float(r2)))


def integer_tiles(codes, t, q, decoder="full", mult=None):
    """T = m_t * X2 per entry (integers, |T| <= 2q m_k), shape (rows, n)."""
    X2 = decode(codes, q, decoder)
    return (X2 * _mult_of(t, mult)[:, :, None]).reshape(codes.shape[0], -1)


def coded_matmul(a_codes, a_t, a_r, qa, base_a, w_codes, w_t, w_r, qw, base_w,
                 decoder_a="full", decoder_w="full", mult_a=None, mult_w=None):
    """C = A_hat W_hat^T from the two coded operands (Alg. 4 for every row pair).

    C_ij = r_Ai r_Wj base_A base_W / 4 * sum_blocks <m_A X2_A, m_W X2_W>.  The integer
    sums are formed with an fp64 matrix product, which is exact because every partial sum
    is an integer below 2^53.  Returns fp64 (M, N).
    """
    TA = integer_tiles(a_codes, a_t, qa, decoder_a, mult_a)
    TW = integer_tiles(w_codes, w_t, qw, decoder_w, mult_w)
    return product_from_tiles(TA, a_r, base_a, TW, w_r, base_w)


def product_from_tiles(TA, a_r, base_a, TW, w_r, base_w):
    """C_ij = r_Ai r_Wj base_A base_W / 4 * sum_l TA_il TW_jl for integer tiles T = m X2
    (``integer_tiles``) and fp32 row scales: the exact integer sums (an fp64 matrix product,
    exact while every partial sum is an integer below 2^53), then the scaling.  fp64 (M, N)."""
    TA = np.asarray(TA).astype(np.float64)
    TW = np.asarray(TW).astype(np.float64)
    bound = float(np.abs(TA).max(initial=0)) * float(np.abs(TW).max(initial=0)) * TA.shape[1]
    assert bound < 2.0 ** 53, "integer sums would not be exact in fp64"
    S = TA @ TW.T
    ra = np.asarray(a_r, np.float32).astype(np.float64)
    rw = np.asarray(w_r, np.float32).astype(np.float64)
    return S * (ra[:, None] * rw[None, :]) * (float(base_a) * float(base_w) / 4.0)
