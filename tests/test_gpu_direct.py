"""GPU parity of two product paths that the other parity tests do not reach.

* nq_matmul, the product that needs no workspace (each workgroup decodes the code words of
  its own rows into on-chip memory and contracts them there): against the oracle's coded
  product (Alg. 4 for every pair of rows, exact integer sums) on ragged shapes, both tile
  configurations (M <= 64 and M > 64), mixed q, both decoders (and the byte decoder at
  q = 16) and beta multiples that need fp16 tiles; and bit for bit against nq_matmul_ex
  where the two sum in the same order (M > 64).
* The 256 x 256 tiles of the decode-once GEMM (bf16, fp16 and int8), which the product
  selects once there is at least one such tile per CU: M = N near 4096 with a short K,
  every output of C against the oracle.

Bar: relative Frobenius error <= 1e-3 and every output within 1e-5 of max |C| (the tiles are
exact integers, only the fp32 accumulation rounds); for the exact int8 contraction every
output within 4e-7 of the oracle's value relative to that value itself.
"""

import numpy as np
import pytest

import workloads
from nq_gpu import oracle_encode_many, upload_coded
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


def _coded_pair(seed, M, N, K, qa, qw, k, decoder="full", mult_a=None, mult_w=None):
    """Oracle-coded A (Student-t rows) and W (N(0, 0.02^2) rows), uploaded, and the oracle's
    product of the two."""
    _, A32 = workloads.random_rows(seed, M, K, dtype="bf16", dist="t4")
    _, W32 = workloads.random_rows(seed + 1000, N, K, dtype="bf16", scale=0.02)
    ka = k if mult_a is None else len(mult_a)
    kw = k if mult_w is None else len(mult_w)
    ba = nestquant.default_base(qa, ka) if mult_a is None else 1.0 / (2 * qa)
    bw = nestquant.default_base(qw, kw) if mult_w is None else 1.0 / (2 * qw)
    ac, ab, ar, TA = oracle_encode_many(A32, qa, ka, ba, decoder, mult_a)
    wc, wb, wr, TW = oracle_encode_many(W32, qw, kw, bw, decoder, mult_w)
    C = nestquant.product_from_tiles(TA, ar, ba, TW, wr, bw)
    dec = 0 if decoder == "full" else 1
    a = upload_coded(ac, ab, ar, M, K, qa, ka, ba, dec, mult=mult_a)
    w = upload_coded(wc, wb, wr, N, K, qw, kw, bw, dec, mult=mult_w)
    return a, w, C


def _check(got, C, exact_int=False):
    g = got.cpu().numpy().astype(np.float64)
    rel = np.linalg.norm(g - C) / max(np.linalg.norm(C), 1e-300)
    assert rel <= (1e-6 if exact_int else MATMUL_RTOL), f"relative Frobenius error {rel}"
    if exact_int:
        bad = np.abs(g - C) > 4e-7 * np.abs(C)
    else:
        bad = np.abs(g - C) > 1e-5 * np.abs(C).max() + 1e-30
    if bad.any():
        i = tuple(np.argwhere(bad)[0])
        pytest.fail(f"{bad.sum()} outputs off; first {i}: got {g[i]!r} want {C[i]!r}")


DIRECT_CASES = [
    # (seed, M, N, K, qa, qw, k, decoder, mult_a, mult_w)
    (200, 1, 1, 8, 14, 14, 4, "full", None, None),
    (201, 16, 14336 // 8, 4096, 14, 14, 4, "full", None, None),      # decode-shaped, 1/8 of N
    (202, 64, 300, 1032, 14, 7, 4, "full", None, None),
    (203, 65, 129, 72, 14, 14, 4, "full", None, None),               # first M of the big tile
    (204, 300, 520, 1160, 16, 14, 4, "full", None, None),
    (205, 513, 260, 264, 7, 7, 4, "full", None, None),
    (206, 40, 300, 1024, 16, 16, 4, "m", None, None),                # byte decoder, q = 16
    (207, 260, 130, 520, 10, 10, 3, "m", None, None),                # packed NestQuantM
    (208, 64, 256, 512, 16, 16, 4, "full", (6, 8, 10, 15), (6, 8, 10, 15)),   # fp16 tiles
    (209, 257, 129, 1032, 16, 14, 4, "full", (6, 8, 10, 15), (2, 3, 5, 8)),   # fp16 tiles
    (210, 33, 65, 64, 14, 14, 1, "full", None, None),
]


@pytest.mark.parametrize("case", DIRECT_CASES,
                         ids=lambda c: f"{c[1]}x{c[2]}x{c[3]}-q{c[4]}/{c[5]}k{c[6]}-{c[7]}"
                                       f"{'-mult' if c[8] else ''}")
def test_matmul_no_workspace_parity(nq, case):
    import torch
    seed, M, N, K, qa, qw, k, decoder, ma, mw = case
    a, w, C = _coded_pair(seed, M, N, K, qa, qw, k, decoder, ma, mw)
    got = nq.matmul_direct(a, w)
    torch.cuda.synchronize()
    _check(got, C)
    if M > 64:
        assert torch.equal(got, nq.matmul(a, w))     # same summation order as decode-once


def test_matmul_no_workspace_strided_output(nq):
    import torch
    a, w, C = _coded_pair(220, 70, 50, 256, 14, 14, 4)
    out = torch.full((70, 64), 7.0, device="cuda")
    nq.matmul_direct(a, w, out=out[:, :50])
    torch.cuda.synchronize()
    _check(out[:, :50], C)
    assert bool((out[:, 50:] == 7.0).all())           # nothing written past N


BIG_TILE_CASES = [
    # (seed, M, N, K, q, k, mult, int8): >= 256 tiles of 256 x 256, short and ragged K
    (230, 4096, 4096, 264, 14, 4, None, False),                     # bf16
    (231, 4000, 3990, 520, 14, 4, None, False),                     # bf16, ragged edges
    (232, 4096, 4096, 264, 14, 4, (6, 8, 10, 16), False),           # fp16 (2q m_k = 448)
    (233, 4096, 4096, 264, 14, 4, None, True),                      # int8 (2q k = 112)
    (234, 4000, 3990, 1032, 7, 4, None, True),                      # int8, ragged edges
]


@pytest.mark.parametrize("case", BIG_TILE_CASES,
                         ids=lambda c: f"{c[1]}x{c[2]}x{c[3]}-q{c[4]}-"
                                       f"{'i8' if c[7] else ('f16' if c[6] else 'bf16')}")
def test_gemm_256x256_tiles(nq, case):
    import torch
    seed, M, N, K, q, k, mult, i8 = case
    a, w, C = _coded_pair(seed, M, N, K, q, q, k, "full", mult, mult)
    mp, np_ = -(-M // 256) * 256, -(-N // 256) * 256
    big, mid = (mp // 256) * (np_ // 256), (mp // 256) * (np_ // 128)
    assert big >= 256 and 2 * -(-big // 256) <= -(-mid // 256)   # the big tile is selected
    got = nq.matmul(a, w, int8=i8)
    torch.cuda.synchronize()
    _check(got, C, exact_int=i8)
