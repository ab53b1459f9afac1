"""GPU tests of nq_encode_matmul, the whole hot path in one call (the encoder writes the
activation's decoded tiles into the product's workspace).

Bar: it must equal nq_encode followed by nq_matmul_ex (or nq_matmul_stages with
NQ_CONTRACT_INT8) bit for bit, codes, beta words, scales and C, since both contract the same
exact integer tiles with the same kernel; and the product must meet the usual oracle bar
(relative Frobenius error <= 1e-3).  Cases cover both product paths (M <= 64 and above),
padding of M and K, fp32 / fp16 / bf16 inputs, both decoders, beta multiples on fp16 tiles,
Opt-beta, the int8 contraction, streamed long rows, zero rows, and the launch that also
carries W's tile decode (rows of 257..2048 blocks, M > 64) with every tile type and decoder.
"""

import numpy as np
import pytest

import workloads
from oracle import layout, nestquant

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


FUSED_CASES = [
    # (seed, M, N, K, dtype, dist, q, k, mult, decoder, strategy, int8)
    (1, 300, 200, 264, "bf16", "t4", 14, 4, None, 0, 0, False),
    (2, 40, 300, 1032, "f16", "normal", 14, 4, None, 0, 0, False),
    (3, 256, 256, 512, "f32", "normal", 16, 4, None, 1, 0, False),
    (4, 130, 70, 72, "bf16", "t4", 16, 4, (6, 8, 10, 15), 0, 0, False),
    (5, 257, 129, 1024, "bf16", "t4", 14, 4, None, 0, 1, False),
    (6, 100, 64, 264, "bf16", "normal", 15, 4, None, 0, 0, True),
    (7, 70, 50, 20000, "bf16", "normal", 14, 4, None, 0, 0, False),
    (8, 16, 100, 4096, "bf16", "t4", 7, 4, None, 1, 0, True),
    (9, 2, 33, 8, "f32", "normal", 14, 4, None, 0, 0, False),
    (10, 64, 128, 128, "bf16", "normal", 12, 3, (2, 5, 9), 1, 1, False),
    # rows of 257..2048 blocks with M > 64: W's tile decode rides in the encoder's launch,
    # for every tile type and decoder variant
    (11, 300, 200, 2056, "bf16", "t4", 14, 4, None, 0, 0, False),
    (12, 130, 77, 4104, "f16", "normal", 16, 4, None, 1, 0, False),
    (13, 96, 300, 3000, "bf16", "t4", 16, 4, (6, 8, 10, 15), 0, 0, False),
    (14, 200, 129, 2304, "bf16", "normal", 15, 4, None, 0, 0, True),
    (15, 65, 64, 16384, "f32", "normal", 7, 4, None, 1, 0, False),
    (16, 80, 50, 8192, "bf16", "t4", 7, 3, (1, 2, 4), 1, 0, True),
    (17, 100, 90, 2560, "bf16", "normal", 16, 3, None, 1, 0, True),
    (18, 70, 40, 4096, "f16", "t4", 16, 4, (5, 9, 20, 40), 1, 0, False),
    # rows of 1025..2048 blocks: W's tile decode workgroups come first in the grid
    (19, 129, 100, 14336, "bf16", "t4", 14, 4, None, 0, 0, True),
    # more than 1024 rows of 257..512 blocks: two-wave encoder workgroups carry W's decode
    (20, 1100, 96, 4096, "bf16", "t4", 14, 4, None, 0, 0, False),
    # one or two activation rows: the product kernel decodes A's codes into LDS itself
    (21, 1, 300, 4104, "bf16", "t4", 16, 4, None, 1, 0, False),
    (22, 2, 130, 2048, "bf16", "normal", 14, 4, None, 0, 0, True),
    (23, 1, 64, 1032, "bf16", "t4", 16, 4, (6, 8, 10, 15), 0, 0, False),
]


@pytest.mark.parametrize("case", FUSED_CASES,
                         ids=lambda c: f"s{c[0]}-{c[1]}x{c[2]}x{c[3]}-{c[4]}-q{c[6]}")
def test_encode_matmul_equals_encode_then_matmul(nq, case):
    import torch
    seed, M, N, K, dtype, dist, q, k, mult, dec, strat, i8 = case
    store, x32 = workloads.random_rows(seed, M, K, dtype=dtype, dist=dist)
    if M > 3:
        store = store.copy()
        store[M // 2] = 0                       # a zero row: r = 0, codes 0, tile 0
        x32 = x32.copy()
        x32[M // 2] = 0
    wstore, w32 = workloads.random_rows(seed + 500, N, K, dtype="bf16", scale=0.02)
    base = None if mult is None else 1.0 / (2 * q)
    w = nq.encode(_dev(wstore, "bf16"), q=q, k=k, decoder=dec)
    x = _dev(store, dtype)
    a1 = nq.encode(x, q=q, k=k, base=base, decoder=dec, strategy=strat, mult=mult)
    c1 = nq.matmul(a1, w, int8=i8)
    a2, c2 = nq.encode_matmul(x, w, q=q, k=k, base=base, decoder=dec, strategy=strat,
                              mult=mult, int8=i8)
    torch.cuda.synchronize()
    assert torch.equal(a1.codes, a2.codes)
    assert torch.equal(a1.beta, a2.beta)
    assert torch.equal(a1.scales, a2.scales)
    assert torch.equal(c1, c2), f"max diff {(c1 - c2).abs().max().item()}"
    # and the oracle's product of the same codes (A from the oracle, W from its own codes)
    dname = "full" if dec == 0 else "m"
    sname = "first" if strat == 0 else "opt"
    bb = nestquant.default_base(q, k) if base is None else base
    ca, ta, ra = nestquant.quantize_rows(x32, q, k, bb, strategy=sname, decoder=dname, mult=mult)
    nbk = K // 8
    wc = layout.unpack_codes(w.codes.cpu().numpy().view(np.uint32).reshape(N, nbk))
    wt = layout.unpack_beta(w.beta.cpu().numpy().view(np.uint32).reshape(N, -1), nbk)
    C = nestquant.coded_matmul(ca, ta, ra, q, bb, wc, wt, w.scales.cpu().numpy(), q, w.base,
                               dname, dname, mult, None)
    g = c2.cpu().numpy().astype(np.float64)
    rel = np.linalg.norm(g - C) / max(np.linalg.norm(C), 1e-300)
    assert rel <= 1e-3, rel


@pytest.mark.parametrize("K", [1024, 2112])
def test_encode_matmul_reuses_its_workspace(nq, K):
    """Two calls in a row on one workspace (a larger product, then a smaller one with more
    padding) give the separate path's results: the padding is cleared on every call (K =
    2112: W's tile decoded inside the encoder's launch)."""
    import torch
    wstore, _ = workloads.random_rows(600, 300, K, dtype="bf16", scale=0.02)
    w = nq.encode(_dev(wstore, "bf16"), 14, 4)
    ws = torch.full((nq.matmul_workspace_size(300, 300, K),), 255, dtype=torch.uint8,
                    device="cuda")
    for M in (300, 70):
        store, _ = workloads.random_rows(601 + M, M, K, dtype="bf16")
        x = _dev(store, "bf16")
        _, c2 = nq.encode_matmul(x, w, 14, 4, workspace=ws)
        c1 = nq.matmul(nq.encode(x, 14, 4), w)
        torch.cuda.synchronize()
        assert torch.equal(c1, c2)


@pytest.mark.parametrize("K", [1024, 2112])
def test_encode_matmul_graph_replays(nq, K):
    """nq_encode_matmul captured in a HIP graph (through torch.cuda.graph) and replayed
    several times, with eager work that changes the input in place between replays: every
    replay equals the eager call on the same input."""
    import torch
    store, _ = workloads.random_rows(610, 300, K, dtype="bf16", dist="t4")
    wstore, _ = workloads.random_rows(611, 260, K, dtype="bf16", scale=0.02)
    w = nq.encode(_dev(wstore, "bf16"), 14, 4)
    x = _dev(store, "bf16").clone()
    ws = torch.empty(nq.matmul_workspace_size(300, 260, K), dtype=torch.uint8, device="cuda")
    codes = torch.empty(300 * (K // 8), dtype=torch.int32, device="cuda")
    beta = torch.empty(300 * ((K // 8 + 15) // 16), dtype=torch.int32, device="cuda")
    scales = torch.empty(300, dtype=torch.float32, device="cuda")
    out = torch.empty(300, 260, device="cuda")
    args = dict(q=14, k=4, out=out, coded_out=(codes, beta, scales), workspace=ws)
    nq.encode_matmul(x, w, **args)                 # warm-up outside the capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        nq.encode_matmul(x, w, **args)
    for rep in range(4):
        x.mul_(1.5 if rep % 2 else -0.75)          # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = (out.clone(), codes.clone(), beta.clone(), scales.clone())
        a_ref, c_ref = nq.encode_matmul(x, w, q=14, k=4)
        torch.cuda.synchronize()
        assert torch.equal(got[0], c_ref)
        assert torch.equal(got[1], a_ref.codes) and torch.equal(got[2], a_ref.beta)
        assert torch.equal(got[3], a_ref.scales)


def test_calls_on_a_side_stream(nq):
    """matmul and encode_matmul queued on a stream other than the current one, with the
    workspace taken from torch's allocator inside the call (and rotate=True's temporary):
    the same results as on the current stream."""
    import torch
    store, _ = workloads.random_rows(620, 300, 2048, dtype="bf16", dist="t4")
    wstore, _ = workloads.random_rows(621, 130, 2048, dtype="bf16", scale=0.02)
    x = _dev(store, "bf16")
    w = nq.encode(_dev(wstore, "bf16"), 14, 4)
    a0, c0 = nq.encode_matmul(x, w, 14, 4)
    m0 = nq.matmul(a0, w)
    r0 = nq.encode(x, 14, 4, rotate=True)
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    a1, c1 = nq.encode_matmul(x, w, 14, 4, stream=side)
    m1 = nq.matmul(a1, w, stream=side)
    r1 = nq.encode(x, 14, 4, rotate=True, stream=side)
    side.synchronize()
    assert torch.equal(c0, c1) and torch.equal(m0, m1)
    assert torch.equal(a0.codes, a1.codes) and torch.equal(r0.codes, r1.codes)
