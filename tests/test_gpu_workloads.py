"""GPU parity at the benchmark workloads' full sizes, through the entry points and launch
configurations that bench.py times.

Coding is row-local (each row's scale, betas and codes depend on that row only), so the
oracle codes the rows in chunks on worker processes (nq_gpu.oracle_encode_many) and its
result for a row is exactly what the GPU must have written for that row of the full matrix;
an entry C_ij of the product depends only on row i of A and row j of W.

* The small case, the decode-shaped layer and the q_proj prefill (16 x 14336 x 4096,
  2048 x 4096 x 4096): every code word, beta word and scale of both operands bit-exact, and
  every output of C within the product bar.
* The down_proj prefill (q = 14 and 7) and the 70B MLP: every code, beta and scale of W and of
  a seeded eighth of A's rows (plus the first and the last row), and every output in those
  rows of C (whole output rows).
* The 2^21 x 128 KV matrix: a seeded eighth of its rows coded and decoded (codes bit-exact,
  decoded values within 1 ulp of fp16).
* The paper's GEMV shape (q = 16, 8192 x 8192, both decoders): the whole of W and all 8192
  outputs.

Product bar: relative Frobenius error <= 1e-3, and every output within 1e-5 of the largest
magnitude of its block (the fp32 accumulation of exact integer products is far tighter).
"""

import numpy as np
import pytest

import workloads
from nq_gpu import oracle_encode_many
from oracle import nestquant

pytestmark = pytest.mark.gpu

MATMUL_RTOL = 1e-3


@pytest.fixture(scope="module")
def nq():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2502_09720_amd as nq
    nq.library()
    return nq


def _dev(store, dtype):
    import torch
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(store).view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(store)).cuda()


def _sample(rng, n, count):
    pick = set(rng.choice(n, size=min(n, count), replace=False).tolist()) | {0, n - 1}
    return np.array(sorted(pick))


def _check_coded(coded, x32, rows, q, k, decoder="full", tiles=True):
    """The GPU's codes, beta words and scales of `rows` (None: every row) against the oracle
    on those rows; returns the oracle's scales and integer tiles of those rows."""
    import torch
    nb = x32.shape[1] // 8
    nbw = (nb + 15) // 16
    codes_d = coded.codes.view(-1, nb)
    beta_d = coded.beta.view(-1, nbw)
    if rows is None:
        codes, beta, scales = codes_d, beta_d, coded.scales
        src = x32
    else:
        idx = torch.from_numpy(rows).cuda()
        codes, beta, scales = codes_d[idx], beta_d[idx], coded.scales[idx]
        src = x32[rows]
    wc, wb, wr, T = oracle_encode_many(src, q, k, decoder=decoder, tiles=tiles)
    got_s = scales.cpu().numpy()
    assert np.array_equal(got_s.view(np.uint32), wr.view(np.uint32)), "scales differ"
    got_c = codes.cpu().numpy().view(np.uint32)
    bad = np.argwhere(got_c != wc)
    assert len(bad) == 0, f"{len(bad)} code words differ, first at {tuple(bad[0])}"
    assert np.array_equal(beta.cpu().numpy().view(np.uint32), wb), "beta words differ"
    # every nibble below q, every beta index below k, over the whole matrix
    assert max(int(((codes_d >> (4 * l)) & 15).max()) for l in range(8)) < q
    assert max(int(((beta_d >> (2 * l)) & 3).max()) for l in range(16)) < k
    return wr, T


def _check_product(got, want):
    got = got.astype(np.float64)
    rel = np.linalg.norm(got - want) / np.linalg.norm(want)
    assert rel <= MATMUL_RTOL, rel
    bad = np.abs(got - want) > 1e-5 * np.abs(want).max()
    assert not bad.any(), f"{bad.sum()} outputs off, first at {tuple(np.argwhere(bad)[0])}"


FULL = {1, 2, 3}                       # workloads checked in full
CASES = [(1, 14), (2, 14), (3, 14), (4, 14), (4, 7), (5, 14)]


@pytest.mark.timeout(900)
@pytest.mark.parametrize("cfg,q", CASES, ids=lambda v: str(v))
def test_workload_full_size(nq, cfg, q):
    """The bench step (nq_encode_matmul with W coded once by nq_encode) at full size."""
    import torch
    c = workloads.WORKLOADS[cfg]
    M, N, K, k = c["M"], c["N"], c["K"], c["k"]
    sa, A32, dt = workloads.operand(cfg, "A")
    sw, W32, _ = workloads.operand(cfg, "W")
    w = nq.encode(_dev(sw, dt), q=q, k=k)
    a, C = nq.encode_matmul(_dev(sa, dt), w, q=q, k=k)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(C).all())
    base = nestquant.default_base(q, k)
    ra = None if cfg in FULL else _sample(np.random.default_rng(7000 + 10 * cfg + q), M, M // 8)
    sca, TA = _check_coded(a, A32, ra, q, k)
    scw, TW = _check_coded(w, W32, None, q, k)
    del A32, W32, sa, sw
    rows = np.arange(M) if ra is None else ra
    # whole output rows, in slices of W's rows to bound the fp64 temporaries
    step = 4096
    for j0 in range(0, N, step):
        want = nestquant.product_from_tiles(TA, sca, base, TW[j0:j0 + step], scw[j0:j0 + step],
                                            base)
        got = C[torch.from_numpy(rows).cuda()][:, j0:j0 + step].cpu().numpy()
        _check_product(got, want)


@pytest.mark.timeout(600)
def test_kv_full_size(nq):
    """The standalone encode / decode of the 2^21 x 128 fp16 matrix at full size: a seeded
    eighth of the rows."""
    import torch
    from nq_gpu import ulp_in
    sx, X32, dt = workloads.operand(5, "X")
    x = _dev(sx, dt)
    coded = nq.encode(x, q=14, k=4)
    dec = nq.decode(coded, torch.float16)
    torch.cuda.synchronize()
    rows = _sample(np.random.default_rng(7100), X32.shape[0], X32.shape[0] // 8)
    from oracle import layout
    wc, wb, r, _ = oracle_encode_many(X32[rows], 14, 4, tiles=False)
    got_c = coded.codes.view(-1, 16)[torch.from_numpy(rows).cuda()].cpu().numpy().view(np.uint32)
    assert np.array_equal(got_c, wc)
    got_b = coded.beta.view(-1, 1)[torch.from_numpy(rows).cuda()].cpu().numpy().view(np.uint32)
    assert np.array_equal(got_b, wb)
    got_s = coded.scales[torch.from_numpy(rows).cuda()].cpu().numpy()
    assert np.array_equal(got_s.view(np.uint32), r.view(np.uint32))
    want = nestquant.decode_rows(layout.unpack_codes(wc), layout.unpack_beta(wb, 16), r, 14,
                                 nestquant.default_base(14, 4))
    got = dec[torch.from_numpy(rows).cuda()].cpu().numpy().astype(np.float64)
    assert not (np.abs(got - want) > ulp_in("f16", want)).any()


@pytest.mark.timeout(600)
@pytest.mark.parametrize("decoder", [1, 0])
def test_gemv_full_size(nq, decoder):
    """The paper's GEMV (q = 16, k = 4; a 1 x 8192 times 8192 x 8192), both decoders: all of W
    and every output."""
    import torch
    n, q, k = 8192, 16, 4
    sa, a32 = workloads.random_rows(8192, 1, n, dtype="bf16")
    sw, w32 = workloads.random_rows(8193, n, n, dtype="bf16", scale=0.02)
    w = nq.encode(_dev(sw, "bf16"), q=q, k=k, decoder=decoder)
    a = nq.encode(_dev(sa, "bf16"), q=q, k=k, decoder=decoder)
    C = nq.matmul(a, w)
    torch.cuda.synchronize()
    name = "full" if decoder == 0 else "m"
    sca, TA = _check_coded(a, a32, None, q, k, name)
    scw, TW = _check_coded(w, w32, None, q, k, name)
    base = nestquant.default_base(q, k)
    want = nestquant.product_from_tiles(TA, sca, base, TW, scw, base)
    _check_product(C.cpu().numpy(), want)
