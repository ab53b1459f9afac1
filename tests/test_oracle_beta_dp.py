"""Pins of the beta-set dynamic program (App. F, Alg. 6) and of the synthetic frontier
(Sec. 6.1, Fig. 3).

* Alg. 6 against brute force: on instances where overload is monotone in beta (a vector
  that overloads at beta_i overloads at every smaller beta), the DP's model is the First-beta
  error, so its value must equal the least First-beta error over all k-subsets whose largest
  beta overloads nothing, and the subset it returns must attain it.
* On any statistics (overload monotone or not) the DP minimizes its own model: its value
  equals the least ``dp_model_loss`` over all admissible k-subsets, found by enumeration,
  and the subset it returns attains it.
* On real E8 statistics (Gaussian 8-vectors, q = 16) overload is nearly monotone; the DP's
  subset is within 1% of the brute-force First-beta optimum there.
* ``block_stats`` and ``first_beta_loss`` against the paper: Table rmse-beta (App. F, q = 16,
  k betas uniform on [0, 10] / q, iid N(0, 1) 8-vectors) is reproduced from the statistics
  alone: sqrt(first_beta_loss / (8 n)) is the First-beta column and the per-vector least
  error over the k betas gives the Opt-beta column.
* The frontier: the information-theoretic bound holds at every point (normalized RMSE >=
  sqrt(Gamma(R))), each rate lies between log2 q and log2 q + log2(k) / 8 (fixed-length
  index), and the error falls as q grows.
* Opt-beta never does worse than First-beta on any block (its choice is the least error).
"""

import math

import numpy as np
import pytest

from oracle import beta_dp, nestquant, theory
from conftest import read_golden


def _monotone_instance(rng, n, m):
    mse = rng.uniform(0.1, 2.0, size=(n, m))
    tau = rng.integers(0, m, size=n)                   # overloads at i < tau_p
    tau[rng.integers(0, n)] = m - 1                     # some vector needs the largest beta
    over = np.arange(m)[None, :] < tau[:, None]
    return mse, over


@pytest.mark.parametrize("seed", range(6))
def test_dp_matches_brute_force_on_monotone_overload(seed):
    rng = np.random.default_rng(seed)
    n, m = int(rng.integers(5, 40)), int(rng.integers(4, 10))
    mse, over = _monotone_instance(rng, n, m)
    for k in range(1, min(m, 4) + 1):
        idx, val = beta_dp.dp_betas(mse, over, k)
        bidx, bval = beta_dp.brute_force_betas(mse, over, k)
        assert bidx is not None and idx is not None
        assert math.isclose(val, bval, rel_tol=1e-12), (k, val, bval)
        assert math.isclose(beta_dp.first_beta_loss(mse, over, idx), val, rel_tol=1e-12)
        assert len(idx) == k and idx == sorted(set(idx))
        assert not over[:, idx[-1]].any()


def test_dp_none_when_every_beta_overloads():
    over = np.ones((3, 4), dtype=bool)
    idx, val = beta_dp.dp_betas(np.ones((3, 4)), over, 2)
    assert idx is None and val == math.inf


def test_dp_on_e8_statistics_is_near_optimal():
    rng = np.random.default_rng(7)
    q = 16
    betas = np.arange(4, 16) / (2.0 * q)                # 2/q .. 7.5/q
    mse, over = beta_dp.block_stats(rng.standard_normal((1500, 8)), betas, q)
    nonmono = (over[:, 1:] & ~over[:, :-1]).any(axis=1).mean()
    assert nonmono < 0.01                               # overload is nearly monotone
    for k in (2, 3):
        idx, _ = beta_dp.dp_betas(mse, over, k)
        _, best = beta_dp.brute_force_betas(mse, over, k)
        assert beta_dp.first_beta_loss(mse, over, idx) <= best * 1.01


def test_frontier_respects_the_bound():
    pts = beta_dp.synthetic_frontier([8, 16], [2, 4], n=192, dim=512, calib=10000, seed=1)
    assert len(pts) == 4
    by = {}
    for q, k, betas, rate, err in pts:
        assert math.log2(q) <= rate <= math.log2(q) + math.log2(k) / 8 + 1e-12
        assert err >= math.sqrt(theory.gamma(rate))
        assert err <= 1.5 * math.sqrt(theory.gamma(rate))
        assert len(betas) == k and (np.diff(betas) > 0).all()
        by[(q, k)] = err
    for k in (2, 4):
        assert by[(16, k)] < by[(8, k)]


def test_exact_sum():
    """Costs are exact sums rounded once: independent of the order of the terms, and right
    where every plain left-to-right order loses the small terms."""
    rng = np.random.default_rng(3)
    ints = rng.integers(0, 1000, 10000).astype(np.float64)
    assert beta_dp.exact_sum(ints) == ints.sum()
    t = np.array([1.0] + [2.0 ** -53] * 127)
    left = 0.0
    for v in t:
        left = left + v
    assert left == 1.0                                   # every tiny term rounds away
    assert beta_dp.exact_sum(t) == 1.0 + 127 * 2.0 ** -53 != left
    assert beta_dp.exact_sum(t[::-1]) == beta_dp.exact_sum(rng.permutation(t))
    assert beta_dp.exact_sum([]) == 0.0


@pytest.mark.parametrize("seed", range(6))
def test_dp_minimizes_its_model_on_any_statistics(seed):
    """Overload drawn at random (not monotone): the DP's value is the least
    dp_model_loss over every admissible k-subset, and its subset attains it."""
    rng = np.random.default_rng(50 + seed)
    n, m = int(rng.integers(5, 40)), int(rng.integers(4, 9))
    mse = rng.uniform(0.1, 2.0, size=(n, m))
    over = rng.random((n, m)) < 0.4
    over[:, -1] = False                                  # the largest beta fits everything
    for k in range(1, min(m, 4) + 1):
        idx, val = beta_dp.dp_betas(mse, over, k)
        bidx, bval = beta_dp.brute_force_betas(mse, over, k, loss=beta_dp.dp_model_loss)
        assert idx is not None and bidx is not None
        assert math.isclose(val, bval, rel_tol=1e-12), (k, val, bval)
        assert math.isclose(beta_dp.dp_model_loss(mse, over, idx), val, rel_tol=1e-12)
        assert len(idx) == k and idx == sorted(set(idx))


@pytest.mark.parametrize("seed", range(3))
def test_model_loss_is_first_beta_loss_when_monotone(seed):
    rng = np.random.default_rng(seed)
    mse, over = _monotone_instance(rng, 60, 7)
    for sub in ([6], [1, 6], [0, 2, 3, 6], [2, 4, 5, 6]):
        assert beta_dp.dp_model_loss(mse, over, sub) == beta_dp.first_beta_loss(mse, over, sub)


def test_block_stats_reproduce_table_rmse_beta():
    """App. F, Table rmse-beta from block_stats alone: sample vectors coded at each of the
    table's k betas (q = 16, beta_t = 10 t / (16 k)); First-beta through first_beta_loss over
    all k betas, Opt-beta as the least error per vector.  Both columns within +-0.0006 of
    the printed values (the table's own rounding plus Monte Carlo noise)."""
    rng = np.random.default_rng(2025)
    v = rng.standard_normal((60000, 8)).astype(np.float32).astype(np.float64)
    q = 16
    for k_s, opt_s, first_s in read_golden("rmse_beta_table.txt"):
        k = int(k_s)
        betas = 10.0 * np.arange(1, k + 1) / k / q
        mse, over = beta_dp.block_stats(v, betas, q)
        first = math.sqrt(beta_dp.first_beta_loss(mse, over, range(k)) / v.size)
        opt = math.sqrt(beta_dp.exact_sum(mse.min(axis=1)) / v.size)
        assert abs(first - float(first_s)) < 6e-4, (k, first, first_s)
        assert abs(opt - float(opt_s)) < 6e-4, (k, opt, opt_s)
        assert opt <= first


def test_entropy_of_usage():
    assert beta_dp.usage_entropy_bits(np.array([1, 2, 3, 4] * 5), 4) == pytest.approx(2.0)
    assert beta_dp.usage_entropy_bits(np.array([3] * 9), 4) == 0.0


@pytest.mark.parametrize("q,k", [(16, 4), (14, 8)])
def test_opt_beta_never_worse_per_block(q, k):
    rng = np.random.default_rng(q + k)
    x = rng.standard_normal((32, 256)).astype(np.float32)
    base = nestquant.default_base(q, k)
    out = {}
    for strat in ("first", "opt"):
        codes, t, r = nestquant.quantize_rows(x, q, k, base, strategy=strat)
        rec = nestquant.decode_rows(codes, t, r, q, base)
        v = x.astype(np.float64) / r.astype(np.float64)[:, None]
        out[strat] = ((rec / r.astype(np.float64)[:, None] - v) ** 2).reshape(32, -1, 8).sum(-1)
    assert (out["opt"] <= out["first"] + 1e-12).all()
    assert (out["opt"] < out["first"]).any()
