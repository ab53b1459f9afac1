"""Choice of the beta set (App. F, Alg. 6) and the synthetic rate-distortion frontier
(Sec. 6.1, Fig. 3).

TEST INFRASTRUCTURE ONLY (see the package docstring).

* ``block_stats``: for sample 8-vectors v (already normalized, as Alg. 3 makes them) and a
  grid of candidate betas, the squared reconstruction error mse[p, i] of v_p coded at
  beta_i and whether that coding overloads (decode(encode(P)) != P, Sec. 4.1).  The lattice
  input is y = fl32(fl32(v) * fl32(1 / beta_i)), one fp32 multiply as in the row quantizer.
* ``dp_betas``: Alg. 6.  dp[i][j] is the least total error of the vectors that do not
  overload at beta_i, coded with beta_i and j - 1 smaller betas under First-beta; the
  transition from the second largest chosen beta s charges the vectors that overload at s
  but not at i with mse[., i].  Index 0 is a virtual beta at which every vector overloads.
  The answer is dp[i][k] for an i at which no vector overloads (readings: the least such
  dp[i][k], the smallest i on a tie; a beta set in which nothing fits is not returned).
  Alg. 6's model equals the First-beta error whenever overload is monotone in beta.
  Reading on the rounding: each cost is the exact sum of its terms over the vectors,
  rounded once to fp64 (no summation order is involved); the recurrence adds costs in
  fp64 as Alg. 6 writes it, and the minima take the first s (and the first i) on exact ties.
* ``dp_model_loss``: the total that Alg. 6's recurrence assigns to a given beta subset (every
  transition's charge, summed exactly), for checking the DP against brute force on any
  statistics.
* ``first_beta_loss``: the total First-beta error of a given beta subset (summed exactly);
  it equals ``dp_model_loss`` when overload is monotone in beta.
* ``synthetic_frontier``: Sec. 6.1's experiment at a small size: for each (q, k) the DP picks
  k betas from the grid {1/2, 1, ..., 25} / q on sample vectors, both matrices are coded with
  them (Alg. 3, First-beta) and multiplied from the codes (Alg. 4); the rate is
  log2 q + H(p) / 8, H the entropy of the betas' usage (the printed formula has the sign of
  the entropy term flipped; read as the entropy), and the error is the root mean squared
  error per entry of A_hat B_hat^T against A B^T for A, B with iid N(0,1) entries, divided by
  sqrt(n) (n = inner dimension; Sec. 6.1's normalization read as the RMSE per entry, which
  the bound E(X^T Y - est)^2 >= n Gamma(R) of Sec. 2.1 compares with sqrt(Gamma(R)),
  ``theory.gamma``).
"""

import itertools
import math

import numpy as np

from .lattice import nearest_e8
from .voronoi import decode, encode_point


def block_stats(v64, betas, q, decoder="full"):
    """(mse (n, m), overload (n, m)) of sample 8-vectors v64 (n, 8) at each beta; the eight
    squares of mse are added in coordinate order."""
    v64 = np.asarray(v64, dtype=np.float64)
    n, m = v64.shape[0], len(betas)
    mse = np.empty((n, m))
    over = np.empty((n, m), dtype=bool)
    v32 = v64.astype(np.float32)
    for i, b in enumerate(betas):
        y = (v32 * np.float32(1.0 / b)).astype(np.float64)
        P = nearest_e8(y)
        X2 = decode(encode_point(P, q), q, decoder)
        over[:, i] = np.any(X2 != P, axis=1)
        acc = np.zeros(n)
        for l in range(8):
            d = b * X2[:, l] / 2.0 - v64[:, l]
            acc = acc + d * d
        mse[:, i] = acc
    return mse, over


def exact_sum(terms):
    """The exact sum of fp64 terms, rounded once to fp64 (math.fsum)."""
    return math.fsum(np.asarray(terms, dtype=np.float64).ravel().tolist())


def dp_betas(mse, over, k):
    """Alg. 6: indices (increasing) of the k betas minimizing the First-beta error, and that
    error; (None, inf) when no beta of the grid is overload-free."""
    n, m = mse.shape
    INF = math.inf
    # virtual beta 0 at which every vector overloads
    ov = np.concatenate([np.ones((n, 1), dtype=bool), over], axis=1)
    ms = np.concatenate([np.zeros((n, 1)), mse], axis=1)
    # cost[s, i]: error of the vectors that overload at beta_s but not at beta_i, coded at
    # beta_i (the same for every j, so computed once)
    cost = np.zeros((m + 1, m + 1))
    for i in range(1, m + 1):
        for s in range(0, i):
            cond = ov[:, s] & ~ov[:, i]
            cost[s, i] = exact_sum(ms[cond, i])
    dp = np.full((m + 1, k + 1), INF)
    frm = np.full((m + 1, k + 1), -1, dtype=np.int64)
    dp[0, 0] = 0.0
    for i in range(1, m + 1):
        for j in range(1, k + 1):
            for s in range(0, i):
                if dp[s, j - 1] == INF:
                    continue
                if dp[i, j] > dp[s, j - 1] + cost[s, i]:
                    dp[i, j] = dp[s, j - 1] + cost[s, i]
                    frm[i, j] = s
    best, pos = INF, -1
    for i in range(1, m + 1):
        if not ov[:, i].any() and dp[i, k] < best:
            best, pos = dp[i, k], i
    if pos < 0:
        return None, INF
    chosen = []
    for j in range(k, 0, -1):
        chosen.append(pos - 1)
        pos = frm[pos, j]
    return sorted(chosen), best


def first_beta_loss(mse, over, subset):
    """Total error of First-beta with the betas `subset` (indices): each vector takes the
    first beta of the subset at which it does not overload, the last one if it overloads at
    all of them (summed exactly)."""
    sub = list(subset)
    ok = ~over[:, sub]
    pick = np.where(ok.any(axis=1), np.argmax(ok, axis=1), len(sub) - 1)
    return exact_sum(mse[np.arange(mse.shape[0]), np.asarray(sub)[pick]])


def dp_model_loss(mse, over, subset):
    """What Alg. 6's recurrence charges for the increasing betas `subset` (s_1 < ... < s_k):
    for each j, the errors at beta_{s_j} of the vectors that overload at s_{j-1} but not at
    s_j (s_0 the virtual beta at which every vector overloads), summed exactly.  inf if the
    largest beta overloads some vector (the DP never returns such a set)."""
    sub = list(subset)
    if over[:, sub[-1]].any():
        return math.inf
    terms = []
    prev = np.ones(mse.shape[0], dtype=bool)
    for s in sub:
        cond = prev & ~over[:, s]
        terms.append(mse[cond, s])
        prev = over[:, s]
    return exact_sum(np.concatenate(terms)) if terms else 0.0


def brute_force_betas(mse, over, k, loss=None):
    """The best k-subset under ``loss`` (default: the First-beta error) among those whose
    largest beta overloads nothing, by enumeration (small grids only); first subset in
    lexicographic order on ties."""
    loss = first_beta_loss if loss is None else loss
    m = mse.shape[1]
    best, arg = math.inf, None
    for sub in itertools.combinations(range(m), k):
        if over[:, sub[-1]].any():
            continue
        val = loss(mse, over, sub)
        if val < best:
            best, arg = val, list(sub)
    return arg, best


def usage_entropy_bits(t, k):
    """Entropy (bits) of the empirical distribution of the beta indices t in 1..k."""
    p = np.bincount(np.asarray(t).ravel(), minlength=k + 1)[1:].astype(np.float64)
    p = p[p > 0] / p.sum()
    return float(-(p * np.log2(p)).sum())


def synthetic_frontier(qs, ks, n=512, dim=1024, calib=10000, seed=0, decoder="full"):
    """Points (q, k, mult, rate bits per entry, normalized RMSE of A_hat B_hat^T) of Sec. 6.1
    at a small size: A, B of shape (n, dim) with iid N(0, 1) entries.  The candidate betas
    are the grid (1/2) {1, ..., 50} / q, i.e. mult_j = j times base = 1 / (2q); the chosen
    set is returned as its multiples."""
    from .nestquant import betas, coded_matmul, quantize_rows
    rng = np.random.default_rng(seed)
    A = rng.standard_normal((n, dim)).astype(np.float32)
    B = rng.standard_normal((n, dim)).astype(np.float32)
    exact = A.astype(np.float64) @ B.astype(np.float64).T
    cal = rng.standard_normal((calib, 8))
    grid = np.arange(1, 51)
    out = []
    for q in qs:
        base = 1.0 / (2 * q)
        mse, over = block_stats(cal, betas(len(grid), base, grid), q, decoder)
        for k in ks:
            idx, _ = dp_betas(mse, over, k)
            if idx is None:
                continue
            mult = grid[idx]
            ca, ta, ra = quantize_rows(A, q, k, base, decoder=decoder, mult=mult)
            cb, tb, rb = quantize_rows(B, q, k, base, decoder=decoder, mult=mult)
            C = coded_matmul(ca, ta, ra, q, base, cb, tb, rb, q, base, decoder, decoder,
                             mult, mult)
            rate = math.log2(q) + usage_entropy_bits(np.concatenate([ta.ravel(), tb.ravel()]),
                                                     k) / 8.0
            err = C - exact
            out.append((q, k, mult, rate, float(np.sqrt((err ** 2).mean() / dim))))
    return out
