"""GPU parity at the benchmark workloads' full sizes, through the entry points and launch
configurations that bench.py times, checked on sampled rows the oracle computes one by one.

Coding is row-local (each row's scale, betas and codes depend on that row only), so the
oracle's codes, beta indices and scales of a sampled row are exactly what the GPU must have
written for that row of the full matrix, and an entry C_ij of the product depends only on
row i of A and row j of W.  Per workload: the rows sampled (seeded, plus the first and the
last row) must match bit for bit; the sampled block of C must meet the product bar
(relative Frobenius error <= 1e-3, and elementwise within 1e-5 of the block's largest
magnitude, the fp32 accumulation of exact integer products being far tighter); and every
code nibble must lie in [0, q) and every beta index in [0, k) over the whole output.
"""

import numpy as np
import pytest

import workloads
from oracle import layout, nestquant

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


def _check_rows(coded, x32, rows, q, k, decoder="full"):
    """The GPU's codes, beta words and scales of `rows` against the oracle on those rows."""
    import torch
    nb = x32.shape[1] // 8
    nbw = (nb + 15) // 16
    idx = torch.from_numpy(rows).cuda()
    codes_d = coded.codes.view(-1, nb)
    beta_d = coded.beta.view(-1, nbw)
    codes = codes_d[idx].cpu().numpy().view(np.uint32)
    beta = beta_d[idx].cpu().numpy().view(np.uint32)
    scales = coded.scales[idx].cpu().numpy()
    c, t, r = nestquant.quantize_rows(x32[rows], q, k, decoder=decoder)
    assert np.array_equal(scales.view(np.uint32), r.view(np.uint32))
    assert np.array_equal(codes, layout.pack_codes(c))
    assert np.array_equal(beta, layout.pack_beta(t))
    # every nibble below q, every beta index below k, over the whole matrix
    assert max(int(((codes_d >> (4 * l)) & 15).max()) for l in range(8)) < q
    assert max(int(((beta_d >> (2 * l)) & 3).max()) for l in range(16)) < k
    return c, t, r


CASES = [(2, 14), (3, 14), (4, 14), (4, 7), (5, 14)]


@pytest.mark.parametrize("cfg,q", CASES, ids=lambda v: str(v))
def test_workload_full_size_sampled(nq, cfg, q):
    """The bench step (nq_encode_matmul with W coded once by nq_encode) at full size."""
    import torch
    c = workloads.WORKLOADS[cfg]
    M, N, K, k = c["M"], c["N"], c["K"], c["k"]
    sa, A32, dt = workloads.operand(cfg, "A")
    sw, W32, _ = workloads.operand(cfg, "W")
    w = nq.encode(_dev(sw, dt), q=q, k=k)
    a, C = nq.encode_matmul(_dev(sa, dt), w, q=q, k=k)
    torch.cuda.synchronize()
    rng = np.random.default_rng(7000 + 10 * cfg + q)
    ra, rw = _sample(rng, M, 10), _sample(rng, N, 10)
    ca, ta, sca = _check_rows(a, A32, ra, q, k)
    cw, tw, scw = _check_rows(w, W32, rw, q, k)
    base = nestquant.default_base(q, k)
    want = nestquant.coded_matmul(ca, ta, sca, q, base, cw, tw, scw, q, base)
    got = C[torch.from_numpy(ra).cuda()][:, torch.from_numpy(rw).cuda()].cpu().numpy()
    got = got.astype(np.float64)
    rel = np.linalg.norm(got - want) / np.linalg.norm(want)
    assert rel <= MATMUL_RTOL, rel
    assert np.all(np.abs(got - want) <= 1e-5 * np.abs(want).max())
    assert bool(torch.isfinite(C).all())


def test_kv_full_size_sampled(nq):
    """The standalone encode / decode of the 2^21 x 128 fp16 matrix at full size."""
    import torch
    from nq_gpu import ulp_in
    sx, X32, dt = workloads.operand(5, "X")
    x = _dev(sx, dt)
    coded = nq.encode(x, q=14, k=4)
    dec = nq.decode(coded, torch.float16)
    torch.cuda.synchronize()
    rows = _sample(np.random.default_rng(7100), X32.shape[0], 2000)
    c, t, r = _check_rows(coded, X32, rows, 14, 4)
    want = nestquant.decode_rows(c, t, r, 14, nestquant.default_base(14, 4))
    got = dec[torch.from_numpy(rows).cuda()].cpu().numpy().astype(np.float64)
    assert not (np.abs(got - want) > ulp_in("f16", want)).any()


@pytest.mark.parametrize("decoder", [1, 0])
def test_gemv_full_size_sampled(nq, decoder):
    """The paper's GEMV (q = 16, k = 4; a 1 x 8192 times 8192 x 8192), both decoders."""
    import torch
    n, q, k = 8192, 16, 4
    sa, a32 = workloads.random_rows(8192, 1, n, dtype="bf16")
    sw, w32 = workloads.random_rows(8193, n, n, dtype="bf16", scale=0.02)
    w = nq.encode(_dev(sw, "bf16"), q=q, k=k, decoder=decoder)
    a = nq.encode(_dev(sa, "bf16"), q=q, k=k, decoder=decoder)
    C = nq.matmul(a, w)
    torch.cuda.synchronize()
    name = "full" if decoder == 0 else "m"
    rw = _sample(np.random.default_rng(7200 + decoder), n, 48)
    ca, ta, sca = _check_rows(a, a32, np.array([0]), q, k, name)
    cw, tw, scw = _check_rows(w, w32, rw, q, k, name)
    base = nestquant.default_base(q, k)
    want = nestquant.coded_matmul(ca, ta, sca, q, base, cw, tw, scw, q, base, name, name)
    got = C[:, torch.from_numpy(rw).cuda()].cpu().numpy().astype(np.float64)
    assert np.linalg.norm(got - want) / np.linalg.norm(want) <= MATMUL_RTOL
    assert np.all(np.abs(got - want) <= 1e-5 * np.abs(want).max())
