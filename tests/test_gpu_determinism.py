"""Run-to-run determinism: every entry point, called twice on the same inputs into fresh
outputs, writes the same bits.  Nothing in the library depends on timing (no atomics on
results, fixed reduction orders), so repeated calls must agree exactly, also at the shapes
the benchmark times."""

import numpy as np
import pytest

import workloads

pytestmark = pytest.mark.gpu


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


def _same(a, b):
    import torch
    return all(torch.equal(x, y) for x, y in zip(a, b))


def test_q_proj_path_is_deterministic(nq):
    import torch
    sa, _, dt = workloads.operand(3, "A")
    sw, _, _ = workloads.operand(3, "W")
    A, W = _dev(sa, dt), _dev(sw, dt)
    runs = []
    for _ in range(2):
        wc = nq.encode(W, q=14, k=4)
        ac = nq.encode(A, q=14, k=4)
        dec = nq.decode(ac, torch.float16)
        c_ex = nq.matmul(ac, wc)
        c_direct = nq.matmul_direct(ac, wc)
        c_i8 = nq.matmul(ac, wc, int8=True)
        a2, c_fused = nq.encode_matmul(A, wc, q=14, k=4)
        rot = nq.rotate(A)
        a3 = nq.encode(A, q=14, k=4, rotate=True)
        opt = nq.encode(A, q=14, k=4, strategy=nq.OPT_BETA)
        torch.cuda.synchronize()
        runs.append([wc.codes, wc.beta, wc.scales, ac.codes, ac.beta, ac.scales, dec, c_ex,
                     c_direct, c_i8, a2.codes, c_fused, rot, a3.codes, a3.beta, opt.codes,
                     opt.beta])
    assert _same(*runs)


def test_skinny_and_kv_paths_are_deterministic(nq):
    import torch
    sa, _, dt = workloads.operand(2, "A")
    sw, _, _ = workloads.operand(2, "W")
    A, W = _dev(sa, dt), _dev(sw, dt)
    x = torch.randn(1 << 16, 128, device="cuda", generator=torch.Generator("cuda").manual_seed(5))
    x = x.to(torch.float16)
    runs = []
    for _ in range(2):
        wc = nq.encode(W, q=14, k=4)
        ac, c = nq.encode_matmul(A, wc, q=14, k=4)
        c2 = nq.matmul_direct(ac, wc)
        kc = nq.encode(x, q=14, k=4)
        kd = nq.decode(kc, torch.float16)
        torch.cuda.synchronize()
        runs.append([wc.codes, ac.codes, c, c2, kc.codes, kc.beta, kc.scales, kd])
    assert _same(*runs)


def test_beta_dp_is_deterministic(nq):
    import torch
    from oracle import nestquant
    q = 14
    v = torch.from_numpy(np.random.default_rng(3).standard_normal((1 << 16, 8)).astype(np.float32)).cuda()
    betas = nestquant.betas(50, 1.0 / (2 * q), np.arange(1, 51))
    runs = []
    for _ in range(2):
        mse, over = nq.beta_stats(v, betas, q)
        chosen, loss = nq.beta_dp(mse, over, 4)
        torch.cuda.synchronize()
        runs.append([mse, over, chosen, loss])
    assert _same(*runs)
