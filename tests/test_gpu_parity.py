"""GPU parity: the HIP path through the C ABI against the oracle, on identical host inputs.

Bar (from the method and its numerics):
* nq_encode: code words, beta words and scales bit-exact;
* nq_decode: every value within 1 ulp of the output type of the oracle's fp64 value;
* nq_matmul: relative Frobenius error <= 1e-3 against the oracle's exact product (bf16
  tiles t*X2 are exact integers; only the fp32 accumulation and the fp32 scale epilogue
  round, so the observed error is ~1e-7).
"""

import numpy as np
import pytest

import workloads
from oracle import nestquant
from nq_gpu import (decoded_to_f64, first_mismatch, oracle_encode, to_device, u32, ulp_in,
                    upload_coded)

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


def check_encode(nq, store, x32, dtype, q, k, base=None, ld_pad=0, decoder="full",
                 strategy="first", mult=None):
    torch = __import__("torch")
    rows, cols = x32.shape
    if ld_pad:
        big = np.zeros((rows, cols + ld_pad), dtype=store.dtype)
        big[:, :cols] = store
        xd = to_device(big, dtype)[:, :cols]
    else:
        xd = to_device(store, dtype)
    got = nq.encode(xd, q=q, k=k, base=base, decoder=0 if decoder == "full" else 1,
                    strategy=nq.FIRST_BETA if strategy == "first" else nq.OPT_BETA, mult=mult)
    torch.cuda.synchronize()
    nb = cols // 8
    gc = u32(got.codes, (rows, nb))
    gb = u32(got.beta, (rows, (nb + 15) // 16))
    gs = got.scales.cpu().numpy()
    oc, ob, os_ = oracle_encode(x32, q, k, base, decoder, strategy, mult)
    assert first_mismatch(gs.view(np.uint32), os_.view(np.uint32)) is None, \
        "scales: " + first_mismatch(gs.view(np.uint32), os_.view(np.uint32))
    m = first_mismatch(gc, oc)
    assert m is None, "codes: " + m
    m = first_mismatch(gb, ob)
    assert m is None, "beta: " + m
    return got


ENCODE_CASES = [
    # (seed, rows, cols, dtype, dist, scale, q, k)
    (1, 64, 512, "f32", "normal", 1.0, 14, 4),
    (2, 37, 8, "bf16", "normal", 1.0, 14, 4),
    (3, 37, 16, "bf16", "normal", 1.0, 14, 4),
    (4, 33, 24, "bf16", "t4", 1.0, 14, 4),
    (5, 20, 120, "f16", "normal", 1.0, 14, 4),
    (6, 20, 136, "bf16", "normal", 0.02, 14, 4),
    (7, 9, 1000, "f32", "t4", 3.0, 7, 4),
    (8, 7, 2056, "bf16", "normal", 1.0, 14, 4),
    (9, 5, 4096, "bf16", "t4", 1.0, 14, 4),
    (10, 3, 14336, "bf16", "normal", 1.0, 14, 4),
    (11, 2, 24576, "f16", "normal", 1.0, 14, 4),
    (12, 2, 40000, "f32", "normal", 1.0, 14, 4),
    (13, 50, 128, "f16", "normal", 1.0, 16, 4),
    (14, 50, 128, "bf16", "t4", 1.0, 3, 2),
    (15, 50, 64, "f32", "uniform", 1.0, 2, 1),
    (16, 50, 96, "bf16", "normal", 1.0, 5, 3),
    (17, 30, 256, "f32", "normal", 1e-30, 14, 4),
    (18, 30, 256, "f32", "normal", 1e30, 12, 4),
    # many short rows: lane groups of 8, 16 and 32 with four blocks per lane (256-block
    # waves), and 33-64-block rows at one row per wave
    (19, 2100, 64, "bf16", "t4", 1.0, 14, 4),
    (20, 1030, 128, "f16", "normal", 1.0, 14, 4),
    (21, 520, 256, "f32", "t4", 1.0, 7, 4),
    (22, 600, 320, "bf16", "normal", 1.0, 16, 4),
]


@pytest.mark.parametrize("case", ENCODE_CASES, ids=lambda c: f"s{c[0]}-{c[1]}x{c[2]}-{c[3]}-q{c[6]}k{c[7]}")
def test_encode_parity(nq, case):
    seed, rows, cols, dtype, dist, scale, q, k = case
    store, x32 = workloads.random_rows(seed, rows, cols, dtype=dtype, scale=scale, dist=dist)
    check_encode(nq, store, x32, dtype, q, k)


def test_encode_strided_rows(nq):
    store, x32 = workloads.random_rows(30, 17, 64, dtype="bf16")
    check_encode(nq, store, x32, "bf16", 14, 4, ld_pad=24)


def test_encode_custom_base(nq):
    store, x32 = workloads.random_rows(31, 40, 128, dtype="f32")
    check_encode(nq, store, x32, "f32", 14, 4, base=0.3)
    check_encode(nq, store, x32, "f32", 10, 2, base=0.11)


def _tie_rows(seed):
    """Rows built to hit the tie rules: quarter/eighth grids, repeated values, constant
    rows, a zero row, single non-zero entries and exact halves after scaling."""
    rng = np.random.default_rng(seed)
    rows = [
        rng.integers(-8, 8, 128) / 4.0,
        rng.integers(-16, 16, 128) / 8.0,
        np.repeat(rng.standard_normal(16), 8),
        np.full(128, 0.75),
        np.zeros(128),
        np.eye(128)[5] * 3.0,
        np.tile([0.5, -0.5, 0.25, 0.0, 1.0, -1.0, 0.125, 2.0], 16),
        rng.choice([-1.0, 1.0], 128),
    ]
    return np.array(rows)


@pytest.mark.parametrize("q,k", [(14, 4), (7, 4), (16, 4), (4, 2), (8, 1)])
def test_encode_ties(nq, q, k):
    x = _tie_rows(q * 10 + k)
    for dtype in ("f32", "bf16"):
        store, x32 = workloads.round_to(x, dtype)
        check_encode(nq, store, x32, dtype, q, k)


def test_encode_outlier_columns(nq):
    store, x32 = workloads.random_rows(40, 24, 1024, dtype="bf16")
    x = x32.astype(np.float64)
    x[:, ::97] *= 20.0
    store, x32 = workloads.round_to(x, "bf16")
    check_encode(nq, store, x32, "bf16", 14, 4)
    check_encode(nq, store, x32, "bf16", 7, 4)


# Opt-beta (App. F): the least-error beta, bit-exact against the oracle's fp64 errors.
# Cases cover every encoder shape (lane groups of 8 .. 256, the streaming kernel beyond
# 2048 blocks), heavy tails (overloaded betas decode far away), ties and both decoders.
OPT_CASES = [c for c in ENCODE_CASES if c[0] in (1, 2, 4, 6, 7, 8, 9, 11, 13, 14, 16)]


@pytest.mark.parametrize("case", OPT_CASES, ids=lambda c: f"s{c[0]}-{c[1]}x{c[2]}-{c[3]}-q{c[6]}k{c[7]}")
def test_encode_opt_beta_parity(nq, case):
    seed, rows, cols, dtype, dist, scale, q, k = case
    store, x32 = workloads.random_rows(seed, rows, cols, dtype=dtype, scale=scale, dist=dist)
    check_encode(nq, store, x32, dtype, q, k, strategy="opt")


@pytest.mark.parametrize("decoder", ["full", "m"])
def test_encode_opt_beta_ties_and_outliers(nq, decoder):
    x = _tie_rows(77)
    store, x32 = workloads.round_to(x, "bf16")
    check_encode(nq, store, x32, "bf16", 16 if decoder == "m" else 14, 4, decoder=decoder,
                 strategy="opt")
    store, x32 = workloads.random_rows(41, 24, 1024, dtype="bf16")
    x = x32.astype(np.float64)
    x[:, ::97] *= 20.0
    store, x32 = workloads.round_to(x, "bf16")
    check_encode(nq, store, x32, "bf16", 16 if decoder == "m" else 14, 4, decoder=decoder,
                 strategy="opt")
    check_encode(nq, store, x32, "bf16", 10, 2, base=0.11, decoder=decoder, strategy="opt")


def test_encode_opt_beta_differs_from_first_beta(nq):
    """The two strategies are different functions: on Gaussian rows some blocks take a
    larger beta under Opt-beta than the first non-overloading one, and the decoded error
    of Opt-beta is never larger per block."""
    torch = __import__("torch")
    store, x32 = workloads.random_rows(42, 64, 1024, dtype="f32")
    xd = to_device(store, "f32")
    a = nq.encode(xd, 14, 4, strategy=nq.FIRST_BETA)
    b = nq.encode(xd, 14, 4, strategy=nq.OPT_BETA)
    da, db = nq.decode(a), nq.decode(b)
    torch.cuda.synchronize()
    assert not np.array_equal(u32(a.beta), u32(b.beta))
    x = x32.astype(np.float64)
    ea = ((da.cpu().numpy().astype(np.float64) - x) ** 2).reshape(64, -1, 8).sum(-1)
    eb = ((db.cpu().numpy().astype(np.float64) - x) ** 2).reshape(64, -1, 8).sum(-1)
    assert (eb <= ea * (1 + 1e-6) + 1e-12).all()
    assert eb.sum() < ea.sum()


def test_encode_non_finite_rows_are_zero(nq):
    torch = __import__("torch")
    x = np.ones((3, 64), np.float32)
    x[0, 3] = np.inf
    x[1, 7] = np.nan
    got = nq.encode(torch.from_numpy(x).cuda(), 14, 4)
    torch.cuda.synchronize()
    codes = u32(got.codes, (3, 8))
    assert not codes[0].any() and not codes[1].any() and codes[2].any()


@pytest.mark.parametrize("out_dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("q,k", [(14, 4), (7, 4), (16, 3), (3, 1)])
def test_decode_parity(nq, out_dtype, q, k):
    torch = __import__("torch")
    store, x32 = workloads.random_rows(50 + q, 45, 520, dtype="bf16", dist="t4")
    base = nestquant.default_base(q, k)
    oc, ob, os_ = oracle_encode(x32, q, k)
    coded = upload_coded(oc, ob, os_, 45, 520, q, k, base)
    tdt = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}[out_dtype]
    out = nq.decode(coded, tdt)
    torch.cuda.synchronize()
    got = decoded_to_f64(out, out_dtype)
    from oracle import layout
    want = nestquant.decode_rows(layout.unpack_codes(oc), layout.unpack_beta(ob, 65), os_, q, base)
    err = np.abs(got - want)
    tol = ulp_in(out_dtype, want)
    bad = err > tol
    assert not bad.any(), f"{bad.sum()} values beyond 1 ulp; worst {err.max()}"


# Rows of a multiple of 16 blocks written without a gap take the decoder's flat addressing
# (beta words and outputs at per-thread constant offsets): 16 blocks (rows stepped with no
# carry), 48 and 512 blocks (with a carry), next to 33 blocks (the general path).
@pytest.mark.parametrize("out_dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("rows,cols", [(1000, 128), (300, 384), (70, 4096), (90, 264)])
def test_decode_parity_row_shapes(nq, out_dtype, rows, cols):
    torch = __import__("torch")
    from oracle import layout
    q, k = 14, 4
    store, x32 = workloads.random_rows(rows + cols, rows, cols, dtype="f16", dist="t4")
    base = nestquant.default_base(q, k)
    oc, ob, os_ = oracle_encode(x32, q, k)
    coded = upload_coded(oc, ob, os_, rows, cols, q, k, base)
    tdt = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}[out_dtype]
    got = decoded_to_f64(nq.decode(coded, tdt), out_dtype)
    want = nestquant.decode_rows(layout.unpack_codes(oc), layout.unpack_beta(ob, cols // 8),
                                 os_, q, base)
    assert np.all(np.abs(got - want) <= ulp_in(out_dtype, want))


def _oracle_product(A32, W32, qa, qw, k):
    ba, bw = nestquant.default_base(qa, k), nestquant.default_base(qw, k)
    ca, ta, ra = nestquant.quantize_rows(A32, qa, k)
    cw, tw, rw = nestquant.quantize_rows(W32, qw, k)
    C = nestquant.coded_matmul(ca, ta, ra, qa, ba, cw, tw, rw, qw, bw)
    from oracle import layout
    A = (layout.pack_codes(ca), layout.pack_beta(ta), ra, ba)
    W = (layout.pack_codes(cw), layout.pack_beta(tw), rw, bw)
    return C, A, W


MATMUL_CASES = [
    # (seed, M, N, K, qa, qw, k)
    (1, 64, 256, 512, 14, 14, 4),
    (2, 1, 1, 8, 14, 14, 4),
    (3, 130, 70, 72, 14, 7, 4),
    (4, 257, 129, 1032, 16, 14, 4),
    (5, 16, 300, 2048, 7, 7, 4),
    (6, 200, 40, 136, 5, 3, 2),
    (7, 33, 65, 64, 14, 14, 1),
    (8, 20, 50, 264, 14, 16, 3),
    (9, 48, 1000, 4096, 14, 14, 4),
    # one or two activation rows: the product kernel decodes A into LDS itself
    (10, 1, 300, 1032, 14, 14, 4),
    (11, 2, 129, 4096, 16, 7, 4),
    (12, 2, 64, 264, 7, 14, 2),
]


@pytest.mark.parametrize("case", MATMUL_CASES, ids=lambda c: f"{c[1]}x{c[2]}x{c[3]}-q{c[4]}/{c[5]}k{c[6]}")
def test_matmul_parity(nq, case):
    torch = __import__("torch")
    seed, M, N, K, qa, qw, k = case
    _, A32 = workloads.random_rows(seed, M, K, dtype="bf16", dist="t4")
    _, W32 = workloads.random_rows(seed + 1000, N, K, dtype="bf16", scale=0.02)
    C, (ac, ab, ar, ba), (wc, wb, wr, bw) = _oracle_product(A32, W32, qa, qw, k)
    a = upload_coded(ac, ab, ar, M, K, qa, k, ba)
    w = upload_coded(wc, wb, wr, N, K, qw, k, bw)
    got = nq.matmul(a, w)
    torch.cuda.synchronize()
    g = got.cpu().numpy().astype(np.float64)
    rel = np.linalg.norm(g - C) / max(np.linalg.norm(C), 1e-300)
    assert rel <= MATMUL_RTOL, f"relative Frobenius error {rel}"
    # elementwise: the fp32 accumulation of exact integer products is far tighter
    assert np.all(np.abs(g - C) <= 1e-5 * np.abs(C).max() + 1e-30)


def test_matmul_strided_output(nq):
    torch = __import__("torch")
    _, A32 = workloads.random_rows(60, 70, 256, dtype="f32")
    _, W32 = workloads.random_rows(61, 50, 256, dtype="f32")
    C, (ac, ab, ar, ba), (wc, wb, wr, bw) = _oracle_product(A32, W32, 14, 14, 4)
    a = upload_coded(ac, ab, ar, 70, 256, 14, 4, ba)
    w = upload_coded(wc, wb, wr, 50, 256, 14, 4, bw)
    buf = torch.full((70, 64), 7.0, device="cuda")
    nq.matmul(a, w, out=buf[:, :50])
    torch.cuda.synchronize()
    g = buf.cpu().numpy()
    assert np.all(g[:, 50:] == 7.0)
    assert np.linalg.norm(g[:, :50] - C) / np.linalg.norm(C) < 1e-6


def test_end_to_end_small_config(nq):
    """The small workload end to end on the GPU (encode both operands, then multiply)."""
    torch = __import__("torch")
    sa, A32, _ = workloads.operand(1, "A")
    sw, W32, _ = workloads.operand(1, "W")
    a = check_encode(nq, sa, A32, "f32", 14, 4)
    w = check_encode(nq, sw, W32, "f32", 14, 4)
    got = nq.matmul(a, w)
    torch.cuda.synchronize()
    C, _, _ = _oracle_product(A32, W32, 14, 14, 4)
    g = got.cpu().numpy().astype(np.float64)
    assert np.linalg.norm(g - C) / np.linalg.norm(C) <= MATMUL_RTOL


def _near_midpoint_rows(n, count=12):
    """Rows (1, b, 0, ..., 0) whose RMS lies within 2^-41 (relative) of an fp32 rounding
    boundary, so that both sides must settle the rounding of the scale exactly."""
    j = np.arange(1, 3_000_000)
    b = (1.0 + j * 2.0 ** -23).astype(np.float32).astype(np.float64)
    r64 = np.sqrt((1.0 + b * b) / n)
    r32 = r64.astype(np.float32)
    up = np.nextafter(r32, np.float32(np.inf)).astype(np.float64)
    dn = np.nextafter(r32, np.float32(-np.inf)).astype(np.float64)
    c = r32.astype(np.float64)
    d = np.minimum(np.abs(r64 - (c + up) / 2), np.abs(r64 - (c + dn) / 2)) / r64
    picks = b[np.nonzero(d < 2.0 ** -41)[0][:count]]
    rows = np.zeros((2 * len(picks), n))
    rng = np.random.default_rng(n)
    for i, bb in enumerate(picks):
        rows[2 * i, 0], rows[2 * i, 1] = 1.0, bb
        rows[2 * i + 1] = rng.standard_normal(n)     # interleave ordinary rows
    return rows


@pytest.mark.parametrize("n", [8, 64, 1024, 4096, 20000])
def test_encode_scale_near_rounding_boundary(nq, n):
    x = _near_midpoint_rows(n)
    store, x32 = workloads.round_to(x, "f32")
    check_encode(nq, store, x32, "f32", 14, 4)


def test_matmul_no_workspace_matches_ex(nq):
    """nq_matmul (no workspace: decodes in the product's tiles) equals nq_matmul_ex (caller
    workspace, decode once) bit for bit for M > 64, where both sum in the same order."""
    torch = __import__("torch")
    _, A32 = workloads.random_rows(70, 300, 256, dtype="bf16")
    _, W32 = workloads.random_rows(71, 200, 256, dtype="bf16", scale=0.02)
    C, (ac, ab, ar, ba), (wc, wb, wr, bw) = _oracle_product(A32, W32, 14, 14, 4)
    a = upload_coded(ac, ab, ar, 300, 256, 14, 4, ba)
    w = upload_coded(wc, wb, wr, 200, 256, 14, 4, bw)
    ref = nq.matmul(a, w)
    out = nq.matmul_direct(a, w)
    torch.cuda.synchronize()
    assert torch.equal(out, ref)
    assert np.linalg.norm(out.cpu().numpy() - C) / np.linalg.norm(C) < 1e-6


@pytest.mark.parametrize("M,N,K", [(40, 300, 512), (300, 200, 256)])
def test_matmul_stages_compose_to_ex(nq, M, N, K):
    """nq_matmul_stages(DECODE) then (CONTRACT) is nq_matmul_ex, bit for bit, on both the
    skinny (M <= 64) and the decode-once path."""
    torch = __import__("torch")
    _, A32 = workloads.random_rows(72, M, K, dtype="bf16")
    _, W32 = workloads.random_rows(73, N, K, dtype="bf16", scale=0.02)
    C, (ac, ab, ar, ba), (wc, wb, wr, bw) = _oracle_product(A32, W32, 14, 14, 4)
    a = upload_coded(ac, ab, ar, M, K, 14, 4, ba)
    w = upload_coded(wc, wb, wr, N, K, 14, 4, bw)
    ref = nq.matmul(a, w)
    ws = torch.empty(nq.matmul_workspace_size(M, N, K), dtype=torch.uint8, device="cuda")
    out = torch.full((M, N), float("nan"), device="cuda")
    nq.matmul(a, w, out=out, workspace=ws, stages=nq.STAGE_DECODE)
    assert torch.isnan(out).all()                      # the decode stage writes no output
    nq.matmul(a, w, out=out, workspace=ws, stages=nq.STAGE_CONTRACT)
    torch.cuda.synchronize()
    assert torch.equal(out, ref)
    assert np.linalg.norm(out.cpu().numpy() - C) / np.linalg.norm(C) < 1e-6


INT8_CASES = [c for c in MATMUL_CASES if c[6] * max(c[4], c[5]) <= 63] + [
    (10, 300, 520, 1160, 14, 14, 4),
    (11, 513, 260, 4096, 15, 15, 4),
    (12, 64, 700, 1032, 15, 14, 4),
]


@pytest.mark.parametrize("case", INT8_CASES, ids=lambda c: f"{c[1]}x{c[2]}x{c[3]}-q{c[4]}/{c[5]}k{c[6]}")
def test_matmul_int8_parity(nq, case):
    """Exact int8 contraction: every inner sum is an exact integer, so each output is within
    a few fp32 roundings of the oracle's value relative to that value itself, even where the
    sum cancels."""
    torch = __import__("torch")
    seed, M, N, K, qa, qw, k = case
    _, A32 = workloads.random_rows(seed, M, K, dtype="bf16", dist="t4")
    _, W32 = workloads.random_rows(seed + 1000, N, K, dtype="bf16", scale=0.02)
    C, (ac, ab, ar, ba), (wc, wb, wr, bw) = _oracle_product(A32, W32, qa, qw, k)
    a = upload_coded(ac, ab, ar, M, K, qa, k, ba)
    w = upload_coded(wc, wb, wr, N, K, qw, k, bw)
    got = nq.matmul(a, w, int8=True)
    torch.cuda.synchronize()
    g = got.cpu().numpy().astype(np.float64)
    rel = np.linalg.norm(g - C) / max(np.linalg.norm(C), 1e-300)
    assert rel <= 1e-6, f"relative Frobenius error {rel}"
    bad = np.abs(g - C) > 4e-7 * np.abs(C)
    if bad.any():
        i = tuple(np.argwhere(bad)[0])
        pytest.fail(f"{bad.sum()} outputs off by more than 4e-7 relative; first {i}: "
                    f"got {g[i]!r} want {C[i]!r}")


@pytest.mark.parametrize("M,N,K", [(40, 300, 1032), (300, 200, 264)])
def test_matmul_int8_tiles_exact(nq, M, N, K):
    """The int8 decode stage writes t * X2 of every block bit-exactly (the oracle's integer
    tiles), zero-padded to the tile grid."""
    torch = __import__("torch")
    _, A32 = workloads.random_rows(74, M, K, dtype="bf16", dist="t4")
    _, W32 = workloads.random_rows(75, N, K, dtype="bf16", scale=0.02)
    _, (ac, ab, ar, ba), (wc, wb, wr, bw) = _oracle_product(A32, W32, 14, 14, 4)
    a = upload_coded(ac, ab, ar, M, K, 14, 4, ba)
    w = upload_coded(wc, wb, wr, N, K, 14, 4, bw)
    ws = torch.zeros(nq.matmul_workspace_size(M, N, K), dtype=torch.uint8, device="cuda")
    out = torch.empty(M, N, device="cuda")
    nq.matmul(a, w, out=out, workspace=ws, stages=nq.STAGE_DECODE, int8=True)
    torch.cuda.synchronize()
    buf = ws.cpu().numpy().view(np.int8)
    kp = -(-K // 128) * 128
    ca, ta, _ = nestquant.quantize_rows(A32, 14, 4)
    TA = nestquant.integer_tiles(ca, ta, 14)
    if M <= 64:
        tiles = [(0, -(-M // 16) * 16, TA)]
    else:
        cw, tw, _ = nestquant.quantize_rows(W32, 14, 4)
        TW = nestquant.integer_tiles(cw, tw, 14)
        mp, np_ = -(-M // 256) * 256, -(-N // 256) * 256
        tiles = [(0, mp, TA), (mp * kp, np_, TW)]
    for off, rows_p, T in tiles:
        got = buf[off:off + rows_p * kp].reshape(rows_p, kp)
        want = np.zeros((rows_p, kp), np.int64)
        want[:T.shape[0], :T.shape[1]] = T
        assert np.array_equal(got.astype(np.int64), want), first_mismatch(got.astype(np.int64), want)


def test_encode_tiny_entries(nq):
    """Entries many orders of magnitude below the row scale (the lattice input is then a
    tiny number of either sign next to exact zeros), in fp32 and bf16."""
    rng = np.random.default_rng(77)
    x = rng.standard_normal((64, 256))
    mask = rng.random((64, 256)) < 0.3
    x[mask] = rng.choice([-1.0, 1.0], mask.sum()) * 10.0 ** rng.uniform(-30, -6, mask.sum())
    x[rng.random((64, 256)) < 0.1] = 0.0
    for dtype in ("f32", "bf16"):
        store, x32 = workloads.round_to(x, dtype)
        check_encode(nq, store, x32, dtype, 14, 4)
        check_encode(nq, store, x32, dtype, 7, 4)


# ------------------------------------------------------------------------------------------
# NestQuantM (App. D): the same encoder, overload judged by the NestQuantM decoder
# ------------------------------------------------------------------------------------------

M_ENCODE_CASES = [
    # (seed, rows, cols, dtype, dist, scale, q, k)
    (40, 64, 512, "f32", "normal", 1.0, 16, 4),
    (41, 200, 128, "f16", "normal", 1.0, 16, 4),
    (42, 37, 8, "bf16", "t4", 1.0, 14, 4),
    (43, 9, 4096, "bf16", "t4", 1.0, 14, 4),
    (44, 3, 20000, "bf16", "normal", 1.0, 16, 4),
    (45, 50, 96, "bf16", "uniform", 1.0, 3, 2),
    (46, 40, 256, "f32", "normal", 1.0, 7, 3),
]


@pytest.mark.parametrize("case", M_ENCODE_CASES, ids=lambda c: f"s{c[0]}-{c[1]}x{c[2]}-{c[3]}-q{c[6]}k{c[7]}")
def test_encode_parity_nestquantm(nq, case):
    seed, rows, cols, dtype, dist, scale, q, k = case
    store, x32 = workloads.random_rows(seed, rows, cols, dtype=dtype, scale=scale, dist=dist)
    check_encode(nq, store, x32, dtype, q, k, decoder="m")


def test_encode_ties_nestquantm(nq):
    x = _tie_rows(47)
    for q, k in [(16, 4), (14, 4), (4, 2)]:
        store, x32 = workloads.round_to(x, "f32")
        check_encode(nq, store, x32, "f32", q, k, decoder="m")


@pytest.mark.parametrize("out", ["f32", "f16", "bf16"])
def test_decode_parity_nestquantm(nq, out):
    torch = __import__("torch")
    _, x32 = workloads.random_rows(48, 100, 264, dtype="bf16")
    codes, t, r = nestquant.quantize_rows(x32, 16, 4, decoder="m")
    from oracle import layout
    coded = upload_coded(layout.pack_codes(codes), layout.pack_beta(t), r, 100, 264, 16, 4,
                         nestquant.default_base(16, 4), 1)
    tdt = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}[out]
    got = decoded_to_f64(nq.decode(coded, tdt), out)
    want = nestquant.decode_rows(codes, t, r, 16, nestquant.default_base(16, 4), decoder="m")
    assert np.all(np.abs(got - want) <= ulp_in(out, want))
    # the NestQuantM decoder really differs from Alg. 5 on these codes
    full = nestquant.decode_rows(codes, t, r, 16, nestquant.default_base(16, 4))
    assert np.any(full != want)


M_MATMUL_CASES = [
    # (seed, M, N, K, q, k, int8)
    (50, 1, 1000, 1024, 16, 4, False),
    (51, 16, 300, 2048, 16, 4, False),
    (52, 200, 130, 520, 16, 4, False),
    (53, 130, 70, 264, 14, 4, True),
    (54, 40, 500, 1032, 15, 4, True),
    (55, 2, 260, 2048, 16, 4, False),
    (56, 1, 100, 1032, 14, 4, True),
]


@pytest.mark.parametrize("case", M_MATMUL_CASES, ids=lambda c: f"{c[1]}x{c[2]}x{c[3]}-q{c[4]}k{c[5]}-{'i8' if c[6] else 'bf16'}")
def test_matmul_parity_nestquantm(nq, case):
    torch = __import__("torch")
    seed, M, N, K, q, k, i8 = case
    _, A32 = workloads.random_rows(seed, M, K, dtype="bf16", dist="t4")
    _, W32 = workloads.random_rows(seed + 1000, N, K, dtype="bf16", scale=0.02)
    b = nestquant.default_base(q, k)
    ca, ta, ra = nestquant.quantize_rows(A32, q, k, decoder="m")
    cw, tw, rw = nestquant.quantize_rows(W32, q, k, decoder="m")
    C = nestquant.coded_matmul(ca, ta, ra, q, b, cw, tw, rw, q, b, "m", "m")
    from oracle import layout
    a = upload_coded(layout.pack_codes(ca), layout.pack_beta(ta), ra, M, K, q, k, b, 1)
    w = upload_coded(layout.pack_codes(cw), layout.pack_beta(tw), rw, N, K, q, k, b, 1)
    got = nq.matmul(a, w, int8=i8)
    torch.cuda.synchronize()
    g = got.cpu().numpy().astype(np.float64)
    rel = np.linalg.norm(g - C) / max(np.linalg.norm(C), 1e-300)
    assert rel <= (1e-6 if i8 else MATMUL_RTOL), f"relative Frobenius error {rel}"


GEMV_EXACT_CASES = [
    # (seed, M, N, K, qa, qw, decoder): one or two activation rows, whose sums are exact int32
    (90, 1, 300, 8192, 16, 16, "full"),
    (91, 2, 129, 4096, 16, 7, "full"),
    (92, 1, 200, 1032, 16, 16, "m"),
    (93, 2, 70, 2056, 14, 14, "m"),
]


@pytest.mark.parametrize("case", GEMV_EXACT_CASES, ids=lambda c: f"{c[1]}x{c[2]}x{c[3]}-q{c[4]}/{c[5]}-{c[6]}")
def test_gemv_exact_integer_sums(nq, case):
    """With one or two activation rows each output is Alg. 4's exact integer sum, rounded
    once to fp32 and scaled by r_A r_W base_A base_W / 4 in fp32 (the scale base_A base_W / 4,
    r_W times it, r_A times that, and the sum times the result: five fp32 roundings in all),
    so every element is within 6 * 2^-24 of the oracle's exact value relatively, however
    much its sum cancels."""
    torch = __import__("torch")
    from oracle import layout
    seed, M, N, K, qa, qw, dec = case
    k = 4
    _, A32 = workloads.random_rows(seed, M, K, dtype="bf16", dist="t4")
    _, W32 = workloads.random_rows(seed + 1000, N, K, dtype="bf16", scale=0.02)
    ba, bw = nestquant.default_base(qa, k), nestquant.default_base(qw, k)
    ca, ta, ra = nestquant.quantize_rows(A32, qa, k, decoder=dec)
    cw, tw, rw = nestquant.quantize_rows(W32, qw, k, decoder=dec)
    C = nestquant.coded_matmul(ca, ta, ra, qa, ba, cw, tw, rw, qw, bw, dec, dec)
    flag = 1 if dec == "m" else 0
    a = upload_coded(layout.pack_codes(ca), layout.pack_beta(ta), ra, M, K, qa, k, ba, flag)
    w = upload_coded(layout.pack_codes(cw), layout.pack_beta(tw), rw, N, K, qw, k, bw, flag)
    got = nq.matmul(a, w)
    torch.cuda.synchronize()
    g = got.cpu().numpy().astype(np.float64)
    err = np.abs(g - C)
    tol = 6 * 2.0 ** -24 * np.abs(C) + 1e-38
    assert np.all(err <= tol), f"worst relative {np.max(err / np.maximum(np.abs(C), 1e-38))}"


# ------------------------------------------------------------------------------------------
# Hadamard rotation (Sec. 5) and rotate-then-encode
# ------------------------------------------------------------------------------------------

ROTATE_CASES = [
    # (seed, rows, cols, dtype, dist)
    (60, 37, 8, "f32", "normal"),
    (61, 300, 128, "f16", "normal"),
    (62, 17, 1024, "bf16", "t4"),
    (63, 9, 4096, "bf16", "t4"),
    (64, 5, 32768, "f32", "normal"),
    (65, 11, 224, "f32", "normal"),
    (66, 7, 1792, "bf16", "normal"),
    (67, 4, 14336, "bf16", "normal"),
    (68, 3, 28672, "f16", "normal"),
    # several rows per workgroup with a ragged last group, the single last stage applied on
    # the way out (16, 256, 4096), and the other pass splits
    (69, 300, 16, "bf16", "normal"),
    (70, 37, 256, "f16", "t4"),
    (71, 13, 512, "f32", "normal"),
    (72, 6, 2048, "bf16", "t4"),
    (73, 5, 8192, "bf16", "normal"),
    (74, 9, 3584, "f16", "normal"),
    (75, 5, 7168, "bf16", "t4"),
]


@pytest.mark.parametrize("case", ROTATE_CASES, ids=lambda c: f"{c[1]}x{c[2]}-{c[3]}")
def test_rotate_parity(nq, case):
    """nq_rotate equals the oracle's fp32 transform bit for bit (same operation order)."""
    torch = __import__("torch")
    from oracle import rotation
    seed, rows, cols, dtype, dist = case
    store, x32 = workloads.random_rows(seed, rows, cols, dtype=dtype, dist=dist)
    x32[0, :] = 0.0
    if dtype == "f32":
        store[0, :] = 0.0
    else:
        store[0, :] = 0
    got = nq.rotate(to_device(store, dtype))
    torch.cuda.synchronize()
    want = rotation.rotate_rows(x32)
    m = first_mismatch(got.cpu().numpy().view(np.uint32), want.view(np.uint32))
    assert m is None, m


def test_rotate_then_encode_parity(nq):
    """Outlier columns, rotated, then coded: codes bit-exact against the oracle's rotation
    followed by its encoder, and the rotation cuts the all-overload blocks."""
    torch = __import__("torch")
    from oracle import rotation
    rng = np.random.default_rng(69)
    x = rng.standard_normal((64, 14336))
    x[:, rng.choice(14336, 143, replace=False)] *= 20.0
    store, x32 = workloads.round_to(x, "bf16")
    y = nq.rotate(to_device(store, "bf16"))
    got = nq.encode(y, q=14, k=4)
    torch.cuda.synchronize()
    yr = rotation.rotate_rows(x32)
    oc, ob, os_ = oracle_encode(yr, 14, 4)
    assert first_mismatch(u32(got.codes, oc.shape), oc) is None
    assert first_mismatch(u32(got.beta, ob.shape), ob) is None
    assert np.array_equal(got.scales.cpu().numpy().view(np.uint32), os_.view(np.uint32))
    _, t_plain, _ = nestquant.quantize_rows(x32[:8], 14, 4)
    _, t_rot, _ = nestquant.quantize_rows(yr[:8], 14, 4)
    assert (t_rot == 4).mean() < (t_plain == 4).mean()


ROTATE_ENCODE_CASES = [
    # (seed, rows, cols, dtype, dist, q, k, decoder, mult): every width the in-LDS rotation
    # holds (4096, 8192, 16384: Sylvester; 3584, 7168, 14336: H_28 mix), 2 / 4 / 8 blocks
    # per lane, all input types, both decoders, beta multiples
    (80, 101, 4096, "bf16", "t4", 14, 4, 0, None),
    (81, 37, 3584, "f16", "normal", 16, 4, 1, None),
    (82, 20, 14336, "bf16", "normal", 7, 4, 0, None),
    (83, 9, 8192, "f32", "t4", 14, 4, 0, (6, 8, 10, 16)),
    (84, 5, 16384, "bf16", "normal", 12, 3, 1, None),
    (85, 3, 7168, "f16", "t4", 15, 2, 0, None),
]


@pytest.mark.parametrize("case", ROTATE_ENCODE_CASES,
                         ids=lambda c: f"s{c[0]}-{c[1]}x{c[2]}-{c[3]}-q{c[5]}")
def test_rotate_encode_equals_rotate_then_encode(nq, case):
    """nq_rotate_encode (rows rotated in LDS, then coded) gives nq_encode(nq_rotate(x))
    bit for bit: codes, beta words and scales, including a zero row."""
    torch = __import__("torch")
    seed, rows, cols, dtype, dist, q, k, dec, mult = case
    store, _ = workloads.random_rows(seed, rows, cols, dtype=dtype, dist=dist)
    store = store.copy()
    store[rows // 2] = 0
    x = to_device(store, dtype)
    base = None if mult is None else 1.0 / (2 * q)
    a1 = nq.encode(nq.rotate(x), q=q, k=k, base=base, decoder=dec, mult=mult)
    a2 = nq.encode(x, q=q, k=k, base=base, decoder=dec, mult=mult, rotate=True)
    torch.cuda.synchronize()
    assert torch.equal(a1.codes, a2.codes)
    assert torch.equal(a1.beta, a2.beta)
    assert torch.equal(a1.scales, a2.scales)
    assert float(a2.scales[rows // 2]) == 0.0


@pytest.mark.parametrize("cols,strategy", [(2048, "first"), (4096, "opt"), (28672, "first")])
def test_rotate_option_falls_back_to_two_passes(nq, cols, strategy):
    """encode(rotate=True) and encode_matmul(rotate=True) where the rotation cannot run in
    the encoder (row widths outside 257..2048 blocks, Opt-beta): nq_rotate, then the plain
    call, with the same results as doing both by hand."""
    torch = __import__("torch")
    from paper_2502_09720_amd import OPT_BETA, FIRST_BETA
    strat = OPT_BETA if strategy == "opt" else FIRST_BETA
    store, _ = workloads.random_rows(89, 7, cols, dtype="bf16", dist="t4")
    x = to_device(store, "bf16")
    y = nq.rotate(x)
    a1 = nq.encode(y, q=14, k=4, strategy=strat)
    a2 = nq.encode(x, q=14, k=4, strategy=strat, rotate=True)
    wstore, _ = workloads.random_rows(90, 70, cols, dtype="bf16")
    wc = nq.encode(nq.rotate(to_device(wstore, "bf16")), q=14, k=4)
    b1, c1 = nq.encode_matmul(y, wc, q=14, k=4, strategy=strat)
    b2, c2 = nq.encode_matmul(x, wc, q=14, k=4, strategy=strat, rotate=True)
    torch.cuda.synchronize()
    assert torch.equal(a1.codes, a2.codes) and torch.equal(a1.beta, a2.beta)
    assert torch.equal(a1.scales, a2.scales)
    assert torch.equal(b1.codes, b2.codes) and torch.equal(c1, c2)


def test_rotate_encode_against_oracle(nq):
    """The fused rotation and coding against the oracle's rotation followed by its encoder."""
    torch = __import__("torch")
    from oracle import rotation
    store, x32 = workloads.random_rows(86, 12, 4096, dtype="bf16", dist="t4")
    got = nq.encode(to_device(store, "bf16"), q=14, k=4, rotate=True)
    torch.cuda.synchronize()
    oc, ob, os_ = oracle_encode(rotation.rotate_rows(x32), 14, 4)
    assert first_mismatch(u32(got.codes, oc.shape), oc) is None
    assert first_mismatch(u32(got.beta, ob.shape), ob) is None
    assert np.array_equal(got.scales.cpu().numpy().view(np.uint32), os_.view(np.uint32))


@pytest.mark.parametrize("M,int8", [(300, False), (300, True), (16, False), (65, True)])
def test_encode_matmul_rotated(nq, M, int8):
    """nq_encode_matmul with NQ_ROTATE_A equals it on the rotated activation, with W coded
    from its rotated rows (A W^T = (A U)(W U)^T), on both product paths."""
    torch = __import__("torch")
    store, _ = workloads.random_rows(87, M, 3584, dtype="bf16", dist="t4")
    wstore, _ = workloads.random_rows(88, 200, 3584, dtype="bf16", scale=0.02)
    x = to_device(store, "bf16")
    q = 15 if int8 else 14
    wc = nq.encode(nq.rotate(to_device(wstore, "bf16")), q=q, k=4)
    a1, c1 = nq.encode_matmul(nq.rotate(x), wc, q=q, k=4, int8=int8)
    a2, c2 = nq.encode_matmul(x, wc, q=q, k=4, int8=int8, rotate=True)
    torch.cuda.synchronize()
    assert torch.equal(a1.codes, a2.codes) and torch.equal(a1.beta, a2.beta)
    assert torch.equal(a1.scales, a2.scales)
    assert torch.equal(c1, c2)


# ---------------------------------------------------------------------------------------
# Beta sets as integer multiples of base (beta_t = m_t base), as the App. F dynamic program
# chooses them from the grid (1/2){1..50}/q = {1..50} / (2q).  Tiles m * X2 use bf16 while
# 2q m_k <= 256, fp16 beyond (exact to 2048), int8 while 2q m_k <= 127.
# ---------------------------------------------------------------------------------------
MULT_ENCODE_CASES = [
    # (seed, rows, cols, dtype, dist, q, mult, strategy, decoder)
    (50, 40, 512, "bf16", "t4", 16, (6, 8, 10, 15), "first", "full"),
    (51, 30, 1000, "f32", "normal", 14, (3, 5, 9), "first", "full"),
    (52, 3, 20000, "bf16", "normal", 14, (2, 3, 5, 8), "first", "full"),
    (53, 40, 256, "bf16", "t4", 16, (6, 8, 10, 15), "opt", "full"),
    (54, 40, 256, "f16", "normal", 16, (5, 7, 11, 50), "first", "m"),
    (55, 64, 64, "f32", "normal", 7, (4,), "first", "full"),
    (56, 9, 4096, "bf16", "t4", 12, (7, 9, 12, 20), "opt", "m"),
]


@pytest.mark.parametrize("case", MULT_ENCODE_CASES,
                         ids=lambda c: f"s{c[0]}-{c[1]}x{c[2]}-q{c[5]}-{c[7]}-{c[8]}")
def test_encode_parity_beta_multiples(nq, case):
    seed, rows, cols, dtype, dist, q, mult, strategy, decoder = case
    store, x32 = workloads.random_rows(seed, rows, cols, dtype=dtype, dist=dist)
    check_encode(nq, store, x32, dtype, q, len(mult), base=1.0 / (2 * q), decoder=decoder,
                 strategy=strategy, mult=mult)


@pytest.mark.parametrize("out_dtype", ["f32", "bf16"])
def test_decode_parity_beta_multiples(nq, out_dtype):
    torch = __import__("torch")
    from oracle import layout
    q, mult = 16, (6, 8, 10, 15)
    base = 1.0 / (2 * q)
    _, x32 = workloads.random_rows(57, 45, 520, dtype="f32", dist="t4")
    oc, ob, os_ = oracle_encode(x32, q, 4, base, mult=mult)
    coded = upload_coded(oc, ob, os_, 45, 520, q, 4, base, mult=mult)
    out = nq.decode(coded, out_dtype={"f32": torch.float32, "bf16": torch.bfloat16}[out_dtype])
    torch.cuda.synchronize()
    got = decoded_to_f64(out, out_dtype)
    want = nestquant.decode_rows(layout.unpack_codes(oc), layout.unpack_beta(ob, 65), os_, q,
                                 base, mult=mult)
    assert not (np.abs(got - want) > ulp_in(out_dtype, want)).any()


def _oracle_product_mult(A32, W32, qa, qw, ma, mw, decoder="full"):
    from oracle import layout
    ba, bw = 1.0 / (2 * qa), 1.0 / (2 * qw)
    ca, ta, ra = nestquant.quantize_rows(A32, qa, len(ma), ba, decoder=decoder, mult=ma)
    cw, tw, rw = nestquant.quantize_rows(W32, qw, len(mw), bw, decoder=decoder, mult=mw)
    C = nestquant.coded_matmul(ca, ta, ra, qa, ba, cw, tw, rw, qw, bw, decoder, decoder, ma, mw)
    A = (layout.pack_codes(ca), layout.pack_beta(ta), ra, ba)
    W = (layout.pack_codes(cw), layout.pack_beta(tw), rw, bw)
    return C, A, W, (ta, tw)


MULT_MATMUL_CASES = [
    # (seed, M, N, K, qa, qw, mult_a, mult_w, int8, decoder)
    (60, 64, 256, 512, 16, 16, (6, 8, 10, 15), (6, 8, 10, 15), False, "full"),     # fp16
    (61, 257, 129, 1032, 16, 14, (6, 8, 10, 15), (2, 3, 5, 8), False, "full"),     # fp16
    (62, 130, 70, 72, 14, 14, (2, 3, 5, 8), (1, 2, 4, 7), False, "full"),          # bf16
    (63, 16, 300, 2048, 14, 14, (2, 3, 5, 8), (1, 2, 3, 4), False, "full"),        # bf16
    (64, 300, 200, 264, 16, 16, (1, 2, 3), (1, 3), True, "full"),                  # int8
    (65, 40, 300, 1032, 16, 16, (5, 7, 11, 50), (6, 8, 10, 15), False, "full"),    # fp16
    (66, 64, 256, 512, 16, 16, (6, 8, 10, 15), (6, 8, 10, 15), False, "m"),        # fp16, bytes
    (67, 300, 130, 264, 16, 16, (6, 8, 10, 15), (3, 4, 5, 7), False, "m"),         # fp16
    (68, 33, 100, 1024, 10, 10, (2, 5, 6), (3, 6), True, "m"),                     # int8
    (69, 1, 200, 1032, 16, 16, (5, 7, 11, 50), (6, 8, 10, 15), False, "full"),     # fp16, M = 1
    (70, 2, 70, 264, 16, 16, (6, 8, 10, 15), (3, 4, 5, 7), False, "m"),            # fp16, M = 2
]


@pytest.mark.parametrize("case", MULT_MATMUL_CASES,
                         ids=lambda c: f"{c[1]}x{c[2]}x{c[3]}-q{c[4]}/{c[5]}-{'i8' if c[8] else 'f'}-{c[9]}")
def test_matmul_parity_beta_multiples(nq, case):
    torch = __import__("torch")
    seed, M, N, K, qa, qw, ma, mw, i8, decoder = case
    _, A32 = workloads.random_rows(seed, M, K, dtype="bf16", dist="t4")
    _, W32 = workloads.random_rows(seed + 1000, N, K, dtype="bf16", scale=0.02)
    C, (ac, ab, ar, ba), (wc, wb, wr, bw), _ = _oracle_product_mult(A32, W32, qa, qw, ma, mw,
                                                                     decoder)
    dec = 0 if decoder == "full" else 1
    a = upload_coded(ac, ab, ar, M, K, qa, len(ma), ba, dec, mult=ma)
    w = upload_coded(wc, wb, wr, N, K, qw, len(mw), bw, dec, mult=mw)
    got = nq.matmul(a, w, int8=i8)
    torch.cuda.synchronize()
    g = got.cpu().numpy().astype(np.float64)
    rel = np.linalg.norm(g - C) / max(np.linalg.norm(C), 1e-300)
    assert rel <= (1e-6 if i8 else MATMUL_RTOL), f"relative Frobenius error {rel}"
    assert np.all(np.abs(g - C) <= 1e-5 * np.abs(C).max() + 1e-30)


@pytest.mark.parametrize("M,N,K", [(40, 300, 1032), (300, 200, 264)])
def test_matmul_fp16_tiles_exact(nq, M, N, K):
    """With multiples beyond bf16's exact range the decode stage writes m * X2 of every
    block as exact fp16 integers (the oracle's integer tiles), zero-padded to the grid."""
    torch = __import__("torch")
    ma, mw, q = (6, 8, 10, 15), (5, 7, 11, 50), 16
    _, A32 = workloads.random_rows(76, M, K, dtype="bf16", dist="t4")
    _, W32 = workloads.random_rows(77, N, K, dtype="bf16", scale=0.02)
    _, (ac, ab, ar, ba), (wc, wb, wr, bw), (ta, tw) = _oracle_product_mult(A32, W32, q, q, ma, mw)
    a = upload_coded(ac, ab, ar, M, K, q, 4, ba, mult=ma)
    w = upload_coded(wc, wb, wr, N, K, q, 4, bw, mult=mw)
    ws = torch.zeros(nq.matmul_workspace_size(M, N, K), dtype=torch.uint8, device="cuda")
    out = torch.empty(M, N, device="cuda")
    nq.matmul(a, w, out=out, workspace=ws, stages=nq.STAGE_DECODE)
    torch.cuda.synchronize()
    buf = ws.cpu().numpy().view(np.float16).astype(np.float64)
    kp = -(-K // 64) * 64
    from oracle import layout
    TA = nestquant.integer_tiles(layout.unpack_codes(ac), ta, q, mult=ma)
    if M <= 64:
        tiles = [(0, -(-M // 16) * 16, TA)]
    else:
        TW = nestquant.integer_tiles(layout.unpack_codes(wc), tw, q, mult=mw)
        assert np.abs(TW).max() > 256          # beyond bf16's exact integers
        mp, np_ = -(-M // 256) * 256, -(-N // 256) * 256
        tiles = [(0, mp, TA), (mp * kp, np_, TW)]
    for off, rows_p, T in tiles:
        got = buf[off:off + rows_p * kp].reshape(rows_p, kp)
        want = np.zeros((rows_p, kp))
        want[:T.shape[0], :T.shape[1]] = T
        assert np.array_equal(got, want), first_mismatch(got, want)


# ---------------------------------------------------------------------------------------
# Maximum row length (K = 65536 = 8192 blocks, the largest the boundary accepts): the
# streamed encoder, the decoder, both product paths and the fused call.
# ---------------------------------------------------------------------------------------
def test_max_cols_encode_decode(nq):
    torch = __import__("torch")
    store, x32 = workloads.random_rows(90, 3, 65536, dtype="bf16", dist="t4")
    got = check_encode(nq, store, x32, "bf16", 14, 4)
    dec = nq.decode(got)
    torch.cuda.synchronize()
    from oracle import layout
    oc, ob, os_ = oracle_encode(x32, 14, 4)
    want = nestquant.decode_rows(layout.unpack_codes(oc), layout.unpack_beta(ob, 8192), os_, 14,
                                 nestquant.default_base(14, 4))
    g = dec.cpu().numpy().astype(np.float64)
    assert not (np.abs(g - want) > ulp_in("f32", want)).any()


@pytest.mark.parametrize("M,N", [(3, 40), (70, 66)])
def test_max_cols_matmul_and_fused(nq, M, N):
    torch = __import__("torch")
    K = 65536
    sa, A32 = workloads.random_rows(91, M, K, dtype="bf16", dist="t4")
    _, W32 = workloads.random_rows(92, N, K, dtype="bf16", scale=0.02)
    C, (ac, ab, ar, ba), (wc, wb, wr, bw) = _oracle_product(A32, W32, 14, 14, 4)
    a = upload_coded(ac, ab, ar, M, K, 14, 4, ba)
    w = upload_coded(wc, wb, wr, N, K, 14, 4, bw)
    got = nq.matmul(a, w)
    _, fused = nq.encode_matmul(to_device(sa, "bf16"), w, 14, 4)
    torch.cuda.synchronize()
    for out in (got, fused):
        g = out.cpu().numpy().astype(np.float64)
        assert np.linalg.norm(g - C) / np.linalg.norm(C) <= MATMUL_RTOL
        assert np.all(np.abs(g - C) <= 1e-5 * np.abs(C).max())
