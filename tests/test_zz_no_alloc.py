"""nq_matmul_static (the product's workspace in the library's static device array, for
callers that cannot allocate) against nq_matmul_ex (caller workspace), through the C ABI.

Both run the same kernels on the same coded operands, so the outputs must agree bit for bit
(well inside the product bar of the other parity tests).  Calls come in a row on one stream,
each smaller than the one before, so every call finds the array holding the previous call's
larger contents; products beyond NQ_STATIC_SCRATCH_BYTES are refused before any launch.
"""

import ctypes

import numpy as np
import pytest

import workloads

pytestmark = pytest.mark.gpu

STATIC_BYTES = 64 << 20


@pytest.fixture(scope="module")
def nq():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2502_09720_amd as nq
    nq.library()
    return nq


def _coded(nq, seed, M, N, K, q=14, k=4):
    import torch
    sa, _ = workloads.random_rows(seed, M, K, dtype="bf16", dist="t4")
    sw, _ = workloads.random_rows(seed + 1, N, K, dtype="bf16", scale=0.02)
    A = torch.from_numpy(sa.view(np.int16)).cuda().view(torch.bfloat16)
    W = torch.from_numpy(sw.view(np.int16)).cuda().view(torch.bfloat16)
    return nq.encode(A, q=q, k=k), nq.encode(W, q=q, k=k)


def _static(nq, a, w, out):
    import torch
    from paper_2502_09720_amd.binding import _params, _stream
    lib = nq.library()
    f = lib.nq_matmul_static
    vp, i64 = ctypes.c_void_p, ctypes.c_int64
    f.argtypes = [vp, vp, vp, vp, i64, vp, vp, vp, vp, i64, i64, vp, i64, vp]
    f.restype = ctypes.c_int
    pa = _params(a.q, a.k, a.base, a.decoder, mult=a.mult)
    pw = _params(w.q, w.k, w.base, w.decoder, mult=w.mult)
    st = f(ctypes.byref(pa), vp(a.codes.data_ptr()), vp(a.beta.data_ptr()),
           vp(a.scales.data_ptr()), a.rows, ctypes.byref(pw), vp(w.codes.data_ptr()),
           vp(w.beta.data_ptr()), vp(w.scales.data_ptr()), w.rows, a.cols,
           vp(out.data_ptr()), out.stride(0), _stream(None))
    return st, lib.nq_last_error().decode()


@pytest.mark.parametrize("shapes", [
    # each call smaller than the one before: decode-once at the 8B q_proj shape (48 MiB of the
    # 64 MiB), a smaller decode-once product, then the skinny path (M <= 64)
    [(2048, 4096, 4096), (300, 520, 1160), (40, 300, 1032)],
])
def test_static_matches_ex_on_consecutive_calls(nq, shapes):
    import torch
    for i, (M, N, K) in enumerate(shapes):
        assert nq.matmul_workspace_size(M, N, K) <= STATIC_BYTES
        a, w = _coded(nq, 900 + 10 * i, M, N, K)
        ref = nq.matmul(a, w)                               # nq_matmul_ex
        out = torch.full((M, N), float("nan"), device="cuda")
        st, msg = _static(nq, a, w, out)
        assert st == 0, msg
        torch.cuda.synchronize()
        assert torch.equal(out, ref), f"call {i} ({M}x{N}x{K}) differs from nq_matmul_ex"


def test_static_refuses_products_beyond_the_array(nq):
    import torch
    M, N, K = 4096, 4096, 8192                               # 128 MiB of workspace
    assert nq.matmul_workspace_size(M, N, K) > STATIC_BYTES
    a, w = _coded(nq, 950, M, N, K)
    out = torch.full((M, N), 7.0, device="cuda")
    st, msg = _static(nq, a, w, out)
    assert st == 2 and "nq_matmul_static" in msg and "workspace" in msg
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())                          # nothing was launched
