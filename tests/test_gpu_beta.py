"""GPU parity of the beta-set statistics and of Alg. 6 (App. F) against the oracle.

Bar: the statistics are bit-exact (the overload flags are integers; each error is the same
eight fp64 operations in the same order).  The dynamic program's costs are sums over the
samples, which the oracle takes exactly (rounded once) and the kernel in a 64-ary tree of
fp64 additions, so near-ties between beta sets may be broken differently.  The kernel's
answer is therefore judged by what it must satisfy: the same solvability; a valid set
(k increasing grid indices whose largest beta overloads no sample); its loss under Alg. 6's
model, summed exactly by the oracle, equal to the oracle's optimum within the summation
bound; and the loss it reports equal to that exact loss within the same bound.  The bound:
in a 64-ary tree of depth d = ceil(log64 n) every non-negative term passes through at most
63 d roundings, and the recurrence adds k costs, so every computed value is within
(63 d + k) 2^-53 of the exact one, relatively; the test allows twice that.
"""

import math

import numpy as np
import pytest

from oracle import beta_dp, nestquant

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def nq():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2502_09720_amd as nq
    nq.library()
    return nq


def _samples(seed, n, kind):
    rng = np.random.default_rng(seed)
    if kind == "normal":
        v = rng.standard_normal((n, 8))
    elif kind == "t4":
        v = rng.standard_t(4, size=(n, 8))
    else:                                    # quarter grid: exact halves after scaling
        v = rng.integers(-12, 13, size=(n, 8)) / 4.0
    return v.astype(np.float32)


def _grid(q, count=50):
    return nestquant.betas(count, 1.0 / (2 * q), np.arange(1, count + 1))


STATS_CASES = [
    # (seed, n, kind, q, decoder, grid size)
    (1, 3000, "normal", 16, "full", 50),
    (2, 2000, "t4", 14, "full", 50),
    (3, 2000, "grid", 7, "full", 30),
    (4, 2000, "normal", 16, "m", 50),
    (5, 1500, "t4", 10, "m", 64),
    (6, 1, "normal", 2, "full", 1),
]


@pytest.mark.parametrize("case", STATS_CASES, ids=lambda c: f"s{c[0]}-{c[2]}-q{c[3]}-{c[4]}-m{c[5]}")
def test_beta_stats_parity(nq, case):
    import torch
    seed, n, kind, q, decoder, m = case
    v = _samples(seed, n, kind)
    betas = _grid(q, m)
    mse, over = nq.beta_stats(torch.from_numpy(v).cuda(), betas, q, 0 if decoder == "full" else 1)
    torch.cuda.synchronize()
    want_mse, want_over = beta_dp.block_stats(v.astype(np.float64), betas, q, decoder)
    got_over = over.cpu().numpy().astype(bool)
    assert np.array_equal(got_over, want_over)
    got = mse.cpu().numpy()
    assert np.array_equal(got.view(np.uint64), want_mse.view(np.uint64)), \
        f"{(got != want_mse).sum()} errors differ"
    if m > 1:
        assert got_over.any() and (~got_over).any()


def _sum_bound(n, k):
    d = 1
    while 64 ** d < max(n, 1):
        d += 1
    return 2.0 * (63 * d + k) * 2.0 ** -53


def _check_dp(chosen, loss, mse, over, k):
    """The kernel's (chosen, loss) against the oracle's exact optimum (module docstring)."""
    n, m = mse.shape
    idx, best = beta_dp.dp_betas(mse, over, k)
    got = chosen.cpu().numpy().tolist()
    got_loss = float(loss.cpu())
    if idx is None:
        assert got == [-1] * k and got_loss == math.inf
        return True
    assert len(got) == k and all(0 <= i < m for i in got) and got == sorted(set(got)), got
    assert not over[:, got[-1]].any(), "the largest chosen beta overloads a sample"
    exact = beta_dp.dp_model_loss(mse, over, got)
    eps = _sum_bound(n, k)
    assert exact <= best * (1 + eps), (got, idx, exact, best)
    assert abs(got_loss - exact) <= eps * exact, (got_loss, exact)
    return got == idx


@pytest.mark.parametrize("q,decoder,kind,solvable", [(16, "full", "normal", True),
                                                     (14, "m", "normal", True),
                                                     (7, "full", "grid", True),
                                                     (12, "full", "t4", False)])
def test_beta_dp_parity(nq, q, decoder, kind, solvable):
    """The kernel's set is optimal under Alg. 6's model within the summation bound, and so
    is its loss; heavy-tailed samples overload even at the largest grid beta, and then both
    report that no set exists."""
    import torch
    v = _samples(10 + q, 4000, kind)
    betas = _grid(q)
    mse, over = nq.beta_stats(torch.from_numpy(v).cuda(), betas, q, 0 if decoder == "full" else 1)
    want_mse, want_over = beta_dp.block_stats(v.astype(np.float64), betas, q, decoder)
    for k in (1, 2, 4, 8):
        chosen, loss = nq.beta_dp(mse, over, k)
        torch.cuda.synchronize()
        assert (beta_dp.dp_betas(want_mse, want_over, k)[0] is not None) == solvable
        _check_dp(chosen, loss, want_mse, want_over, k)


def test_beta_dp_on_monotone_instances(nq):
    """Synthetic statistics with monotone overload (where Alg. 6's model is the First-beta
    error): the kernel's set is optimal within the summation bound."""
    import torch
    same = total = 0
    for seed in range(5):
        rng = np.random.default_rng(100 + seed)
        n, m = int(rng.integers(50, 300)), int(rng.integers(5, 64))
        mse = rng.uniform(0.1, 2.0, size=(n, m))
        tau = rng.integers(0, m, size=n)
        over = np.arange(m)[None, :] < tau[:, None]
        md, od = torch.from_numpy(mse).cuda(), torch.from_numpy(over.astype(np.uint8)).cuda()
        for k in sorted({1, 2, min(4, m), min(7, m)}):
            chosen, loss = nq.beta_dp(md, od, k)
            torch.cuda.synchronize()
            same += _check_dp(chosen, loss, mse, over, k)
            total += 1
    print(f"kernel's set equal to the oracle's on {same} of {total} instances")


def test_beta_dp_large_sample(nq):
    """2^16 Gaussian samples, 50 grid betas: trees of depth 3 on the kernel's side (the
    frontier's 2^18 calibration samples also take depth 3)."""
    import torch
    q = 14
    v = _samples(77, 1 << 16, "normal")
    betas = _grid(q)
    mse, over = nq.beta_stats(torch.from_numpy(v).cuda(), betas, q)
    want_mse, want_over = beta_dp.block_stats(v.astype(np.float64), betas, q)
    assert np.array_equal(over.cpu().numpy().astype(bool), want_over)
    for k in (2, 4):
        chosen, loss = nq.beta_dp(mse, over, k)
        torch.cuda.synchronize()
        _check_dp(chosen, loss, want_mse, want_over, k)


def test_beta_dp_every_beta_overloads(nq):
    import torch
    over = np.ones((20, 6), dtype=np.uint8)
    over[:, 5] = 0
    over[3, 5] = 1                                  # even the largest beta overloads one
    mse = np.ones((20, 6))
    chosen, loss = nq.beta_dp(torch.from_numpy(mse).cuda(), torch.from_numpy(over).cuda(), 3)
    torch.cuda.synchronize()
    assert chosen.cpu().numpy().tolist() == [-1, -1, -1]
    assert float(loss.cpu()) == float("inf")
    assert beta_dp.dp_betas(mse, over.astype(bool), 3) == (None, float("inf"))


def test_beta_dp_no_samples(nq):
    import torch
    e = torch.empty(0, 7, dtype=torch.float64, device="cuda")
    o = torch.empty(0, 7, dtype=torch.uint8, device="cuda")
    chosen, loss = nq.beta_dp(e, o, 3)
    torch.cuda.synchronize()
    idx, val = beta_dp.dp_betas(np.zeros((0, 7)), np.zeros((0, 7), dtype=bool), 3)
    assert chosen.cpu().numpy().tolist() == idx == [0, 1, 2]
    assert float(loss.cpu()) == val == 0.0


def test_chosen_betas_drive_the_encoder(nq):
    """The DP's indices on the grid {1..50} / (2q) are the encoder's multiples of base
    1 / (2q): coding rows with them matches the oracle bit for bit."""
    import torch
    import workloads
    from nq_gpu import oracle_encode, u32
    q, k = 14, 4
    v = _samples(31, 4000, "normal")
    mse, over = nq.beta_stats(torch.from_numpy(v).cuda(), _grid(q), q)
    chosen, _ = nq.beta_dp(mse, over, k)
    mult = tuple(int(i) + 1 for i in chosen.cpu().numpy())
    store, x32 = workloads.random_rows(32, 48, 1024, dtype="bf16")
    xd = torch.from_numpy(store.view(np.int16)).cuda().view(torch.bfloat16)
    got = nq.encode(xd, q=q, k=k, base=1.0 / (2 * q), mult=mult)
    torch.cuda.synchronize()
    oc, ob, os_ = oracle_encode(x32, q, k, 1.0 / (2 * q), mult=mult)
    assert np.array_equal(u32(got.codes, oc.shape), oc)
    assert np.array_equal(u32(got.beta, ob.shape), ob)
