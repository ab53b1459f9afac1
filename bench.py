#!/usr/bin/env python3
"""Benchmark of the NestQuant coded-GEMM hot path on one MI355X.

One step = one pass of the whole hot path over one batch of the Llama-3-8B q_proj prefill
workload: nq_encode_matmul, i.e. the coding of the activations A (2048 x 4096 bf16,
Student-t(4)) and the product of the coded A with the coded weight W (4096 x 4096 bf16,
N(0, 0.02^2)), q = 14, k = 4, in one call.  W is a weight: it is coded once, before timing.  Inputs are resident in HBM when
the timed region starts; A is rotated over enough copies (> 512 MB) that the 256 MB
Infinity Cache cannot serve the encoder's reads.

Prints one JSON line (see the "value" fields below).  Kernel durations come from HIP events
recorded on the stream the kernels run on.
"""

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0     # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
INT8_PEAK_TOPS = 5000.0    # MI355X dense int8 MFMA

METRIC = "nq_matmul TFLOP/s + nq_encode GB/s (q=14,k=4) at Llama-3-8B prefill shapes"


def stats(ms):
    """mean, median and min of per-call event times (ms)."""
    a = np.asarray(ms, dtype=np.float64)
    return {"mean_ms": float(a.mean()), "median_ms": float(np.median(a)), "min_ms": float(a.min())}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=100,
                    help="untimed steps first (the first ~10 ms of back-to-back steps run "
                         "slower, about 120 against 104 us per q_proj step)")
    ap.add_argument("--workload", type=int, default=3, help="workload id (see workloads.py)")
    ap.add_argument("--q", type=int, default=None, help="override q (workload 4 has q=7 too)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-kv", action="store_true",
                    help="leave out the standalone encode / decode of the 2^28-entry KV matrix")
    ap.add_argument("--graph", action="store_true",
                    help="replay a captured HIP graph of the step instead of launching its "
                         "kernels directly (slower on these boxes)")
    ap.add_argument("--kv", action="store_true",
                    help="standalone nq_encode / nq_decode of the 2^28-entry fp16 KV-like "
                         "matrix (2^21 rows of 128) against the HBM roofline")
    ap.add_argument("--gemv", action="store_true",
                    help="the paper's GEMV: one coded 8192-vector times a coded 8192 x 8192 "
                         "matrix, q=16, k=4, NestQuantM and full decoders, against HBM")
    ap.add_argument("--frontier", action="store_true",
                    help="Sec. 6.1 on the GPU: A, B 4096 x 4096 iid N(0,1); for each (q, k) "
                         "the beta set chosen by Alg. 6 from (1/2){1..50}/q, both coded, "
                         "multiplied from the codes; rate and RMSE against sqrt(Gamma(R))")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="calibration only: time a plain device-to-device copy of this many "
                         "bytes (the reference for the HBM byte counters)")
    return ap.parse_args()


def gemv_roofline(args):
    """The paper's GEMV (App. E runtime table): C = a W^T with a 1 x 8192 and W 8192 x 8192,
    both NestQuant-coded at q=16, k=4 (4.25 bits per entry), with the NestQuantM decoder (the
    paper's kernel) and with the full decoder.  W ~ N(0, 0.02^2) bf16 and a ~ N(0, 1) bf16,
    drawn from seeded streams; W is rotated over enough copies (> 256 MB) that the Infinity
    Cache cannot hold it.  Bytes = coded W + coded a + fp32 output."""
    import numpy as np
    import torch
    import workloads
    import paper_2502_09720_amd as nq
    dev = torch.device("cuda:0")
    n = 8192
    q, k = 16, 4
    sa, _ = workloads.random_rows(8192, 1, n, dtype="bf16")
    sw, _ = workloads.random_rows(8193, n, n, dtype="bf16", scale=0.02)
    A = torch.from_numpy(sa.view(np.int16)).to(dev).view(torch.bfloat16)
    W = torch.from_numpy(sw.view(np.int16)).to(dev).view(torch.bfloat16)
    nb = n // 8
    coded_w = n * nb * 4 + n * ((nb + 15) // 16) * 4 + n * 4
    nbuf = -(-256 * 2**20 // coded_w) + 1
    res = {}
    for name, dec in (("nestquantm", nq.DECODER_M), ("full", nq.DECODER_FULL)):
        ac = nq.encode(A, q=q, k=k, decoder=dec)
        wcs = [nq.encode(W, q=q, k=k, decoder=dec) for _ in range(nbuf)]
        C = torch.empty(1, n, dtype=torch.float32, device=dev)
        ws = torch.empty(nq.matmul_workspace_size(1, n, n), dtype=torch.uint8, device=dev)
        for i in range(args.warmup):
            nq.matmul(ac, wcs[i % nbuf], out=C, workspace=ws)
        torch.cuda.synchronize()
        # back-to-back calls, timed as a whole: per-call event pairs would also time the
        # host's gap between two launches (a few microseconds, more than this product's
        # launch-to-launch overhead on the GPU)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        h0 = time.perf_counter()
        for i in range(args.steps):
            nq.matmul(ac, wcs[i % nbuf], out=C, workspace=ws)
        host_us = (time.perf_counter() - h0) / args.steps * 1e6   # issue time per call
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) / args.steps * 1e3
        byts = coded_w + nb * 4 + 4 + 4 + n * 4
        res[name] = {"us": us, "GBps": byts / (us * 1e-6) / 1e9,
                     "hbm_frac": byts / (us * 1e-6) / 1e9 / HBM_PEAK_GBPS,
                     "bytes": byts, "w_copies": nbuf, "host_issue_us": host_us,
                     "launches": "one (the vector is decoded inside the product kernel)"}
        del wcs
    print(json.dumps({"metric": "coded GEMV time, 8192 x 8192, q=16, k=4 (4.25 bits/entry)",
                      "unit": "us", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
                      "dtype": "bf16", "data": "synthetic",
                      "config": {"workload": "GEMV a (1x8192) W^T (8192x8192), W N(0,0.02^2)"},
                      "results": res,
                      "paper_context": "NestQuantM 60 us on an NVIDIA A100 (App. E table)"}))


def gamma_bound(R):
    """Gamma(R) (Sec. 2.1): the least inner-product distortion per entry at rate R for iid
    N(0, 1) vectors: 2 2^-2R - 2^-4R above R*, the tangent line from (0, 1) below it."""
    phi = lambda x: 2.0 * 2.0 ** (-2 * x) - 2.0 ** (-4 * x)               # noqa: E731
    dphi = lambda x: np.log(2) * (-4.0 * 2.0 ** (-2 * x) + 4.0 * 2.0 ** (-4 * x))  # noqa: E731
    lo, hi = 0.1, 3.0
    for _ in range(100):                       # touching point: (phi(R) - 1) / R = phi'(R)
        mid = 0.5 * (lo + hi)
        if ((phi(mid) - 1.0) / mid - dphi(mid)) * ((phi(lo) - 1.0) / lo - dphi(lo)) > 0:
            lo = mid
        else:
            hi = mid
    rs = 0.5 * (lo + hi)
    return phi(R) if R >= rs else 1.0 - (1.0 - phi(rs)) * R / rs


def frontier(args):
    """Sec. 6.1 (Fig. 3) at the paper's size on the GPU.  For each (q, k): nq_beta_stats of
    2^18 N(0, 1) sample 8-vectors at the 50 grid betas {1..50} / (2q), nq_beta_dp for k of
    them, nq_encode of A and B with those multiples (base 1 / (2q)), nq_matmul, and the
    normalized RMSE sqrt(mean((A_hat B_hat^T - A B^T)^2) / n) against sqrt(Gamma(R)) at the
    entropy rate R = log2 q + H(beta usage) / 8.  The same (q, k) with the uniform grid
    (base 10 / (kq)) is reported beside it.  One JSON line per point, then a summary line."""
    import torch
    import paper_2502_09720_amd as nq
    nq.library()
    dev = torch.device("cuda")
    n = 4096
    g = torch.Generator(device=dev)
    g.manual_seed(61)
    A = torch.randn(n, n, generator=g, device=dev, dtype=torch.float32)
    B = torch.randn(n, n, generator=g, device=dev, dtype=torch.float32)
    cal = torch.randn(1 << 18, 8, generator=g, device=dev, dtype=torch.float32)
    exact = A.double() @ B.double().T
    grid = np.arange(1, 51)

    def usage_bits(c, k):
        words = c.beta
        idx = torch.stack([(words >> (2 * j)) & 3 for j in range(16)], 1).reshape(c.rows, -1)
        idx = idx[:, : c.cols // 8].reshape(-1).long()
        p = torch.bincount(idx, minlength=4)[:k].double()
        p = p[p > 0] / p.sum()
        return float(-(p * torch.log2(p)).sum())

    def point(q, k, base, mult):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        ev[0].record()
        a = nq.encode(A, q=q, k=k, base=base, mult=mult)
        ev[1].record()
        b = nq.encode(B, q=q, k=k, base=base, mult=mult)
        ev[2].record()
        C = nq.matmul(a, b)
        ev[3].record()
        torch.cuda.synchronize()
        err = float(torch.sqrt(((C.double() - exact) ** 2).mean() / n))
        h = 0.5 * (usage_bits(a, k) + usage_bits(b, k))
        rate = float(np.log2(q) + h / 8.0)
        return {"rate_bits": rate, "rate_fixed_bits": float(np.log2(q) + np.log2(k) / 8),
                "rmse": err, "sqrt_gamma": float(np.sqrt(gamma_bound(rate))),
                "encode_ms": ev[0].elapsed_time(ev[1]), "matmul_ms": ev[2].elapsed_time(ev[3])}

    pts = []
    for q in (3, 4, 5, 6, 7, 8, 10, 12, 14, 16):
        betas = grid / (2.0 * q)
        e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
        e0.record()
        mse, over = nq.beta_stats(cal, betas, q)
        e1.record()
        for k in (1, 2, 3, 4):
            e1b = torch.cuda.Event(enable_timing=True)
            e1b.record()
            chosen, loss = nq.beta_dp(mse, over, k)
            e2.record()
            torch.cuda.synchronize()
            idx = chosen.cpu().numpy()
            if (idx < 0).any():
                continue
            mult = tuple(int(i) + 1 for i in idx)
            row = {"q": q, "k": k, "betas_times_2q": list(mult),
                   "beta_stats_ms": e0.elapsed_time(e1), "beta_dp_ms": e1b.elapsed_time(e2)}
            row["dp"] = point(q, k, 1.0 / (2 * q), mult)
            row["uniform"] = point(q, k, 10.0 / (k * q), None)
            pts.append(row)
            print(json.dumps(row), flush=True)
    # efficient frontier of the DP points: no other point has lower rate and lower error
    front = []
    for r in pts:
        d = r["dp"]
        if not any(o["dp"]["rate_bits"] <= d["rate_bits"] and o["dp"]["rmse"] < d["rmse"]
                   and o is not r for o in pts):
            front.append((r["q"], r["k"], round(d["rate_bits"], 4), round(d["rmse"], 5),
                          round(d["rmse"] / d["sqrt_gamma"], 3)))
    print(json.dumps({"frontier": sorted(front, key=lambda t: t[2]),
                      "columns": ["q", "k", "rate_bits", "rmse", "rmse_over_sqrt_gamma"],
                      "n": n, "samples": 1 << 18, "data": "synthetic iid N(0,1)"}))


def copy_calibration(args):
    """A plain device copy of known size, for scaling FETCH_SIZE / WRITE_SIZE readings."""
    import torch
    n = args.copy_bytes
    src = torch.ones(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(args.warmup):
        dst.copy_(src)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    print(json.dumps({"metric": "device copy", "bytes_read": n, "bytes_written": n, "ms": ms,
                      "GBps": 2 * n / (ms * 1e-3) / 1e9}))


def kv_measure(steps, warmup):
    """nq_encode and nq_decode of X (2^21 x 128 fp16 N(0,1)) against 8 TB/s: per call the
    algorithmic bytes (fp16 in or out, codes, beta words, scales) over its event time.  X is
    512 MiB, twice the Infinity Cache, so every call streams it from HBM."""
    import torch
    import workloads
    import paper_2502_09720_amd as nq

    c = workloads.WORKLOADS[5]
    rows, cols = c["X_rows"], c["X_cols"]
    dev = torch.device("cuda:0")
    X = torch.empty(rows, cols, dtype=torch.float16, device=dev)
    step = 1 << 17
    for r0 in range(0, rows, step):
        st, _, _ = workloads.operand(5, "X", row_range=(r0, min(rows, r0 + step)))
        X[r0:r0 + len(st)] = torch.from_numpy(st).to(dev)
    q, k = 14, 4
    coded = nq.encode(X, q=q, k=k)
    out = torch.empty_like(X)
    nb = cols // 8
    io = rows * cols * 2
    coded_bytes = rows * nb * 4 + rows * ((nb + 15) // 16) * 4 + rows * 4
    res = {}
    for name, fn in (("nq_encode", lambda: nq.encode(X, q=q, k=k, out=(coded.codes, coded.beta,
                                                                        coded.scales))),
                     ("nq_decode", lambda: nq.decode(coded, torch.float16, out=out))):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(steps)]
        for i in range(steps):
            ev[i][0].record()
            fn()
            ev[i][1].record()
        torch.cuda.synchronize()
        t = stats([e[0].elapsed_time(e[1]) for e in ev])
        gbps = (io + coded_bytes) / (t["median_ms"] * 1e-3) / 1e9
        res[name] = dict(t, GBps=gbps, hbm_frac=gbps / HBM_PEAK_GBPS, bytes=io + coded_bytes)
    del X, out, coded
    return res


def kv_roofline(args):
    res = kv_measure(args.steps, args.warmup)
    print(json.dumps({"metric": "nq_encode / nq_decode GB/s, 2^28 fp16 entries in rows of 128",
                      "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
                      "dtype": "f16", "data": "synthetic",
                      "config": {"workload": "KV-like 2^21 x 128 fp16 N(0,1), q=14, k=4"},
                      "results": res}))


def gemm_traffic(cfg, q):
    """HBM bytes per gemm_kernel launch from the committed counter summary, or None.

    The summary records FETCH_SIZE and WRITE_SIZE of one launch (rocprofv3 --pmc), the same
    counters for a device-to-device copy of known size (the calibration factor), and the
    SHA-256 of the kernel source the counters were taken on: once that source changes, the
    figure no longer describes the kernel and None is reported."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"gemm_kernel_workload{cfg}_traffic.md")
    src = os.path.join(ROOT, "paper_2502_09720_amd", "csrc", "nq_gemm.hip")
    if not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if line.startswith("- ") and ":" in line:
            key, val = line[2:].split(":", 1)
            fields[key.strip()] = val.strip().strip("`")
    digest = hashlib.sha256(open(src, "rb").read()).hexdigest()
    if fields.get("kernel source sha256") != digest or fields.get("q") != str(q):
        return None
    return float(fields["traffic bytes per launch"])


def algorithmic(M, N, K, in_bytes):
    nb = K // 8
    nbw = (nb + 15) // 16
    coded = lambda rows: rows * nb * 4 + rows * nbw * 4 + rows * 4  # noqa: E731
    enc_bytes = M * K * in_bytes + coded(M)
    mm_bytes = coded(M) + coded(N) + M * N * 4
    flops = 2.0 * M * N * K
    return enc_bytes, mm_bytes, flops


def cpu_baseline(cfg, q, k, flops_full, min_seconds=10.0, max_reps=5):
    """The oracle, as it stands, on the whole step of the workload, repeated until about
    min_seconds of CPU time have been measured: encode of A, decode of A and W into integer
    tiles, and the exact fp64 product with the scale epilogue.  W's coding is excluded, as
    on the GPU (W is a weight, coded once)."""
    import numpy as np
    import workloads
    from oracle import nestquant
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([d.get("num_threads", 1) for d in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        blas_threads = 1
    c = workloads.WORKLOADS[cfg]
    M, N, K = c["M"], c["N"], c["K"]
    _, A32, _ = workloads.operand(cfg, "A")
    _, W32, _ = workloads.operand(cfg, "W")
    base = nestquant.default_base(q, k)
    cw, tw, rw = nestquant.quantize_rows(W32, q, k)
    times, enc_times = [], []
    while len(times) < max_reps and (len(times) < 2 or sum(times) < min_seconds):
        t0 = time.perf_counter()
        ca, ta, ra = nestquant.quantize_rows(A32, q, k)
        enc_times.append(time.perf_counter() - t0)
        TA = nestquant.integer_tiles(ca, ta, q).astype(np.float64)
        TW = nestquant.integer_tiles(cw, tw, q).astype(np.float64)
        S = TA @ TW.T
        _ = S * (ra.astype(np.float64)[:, None] * rw.astype(np.float64)[None, :]) * (base * base / 4)
        times.append(time.perf_counter() - t0)
        del TA, TW, S
    step = float(np.mean(times))
    enc = float(np.mean(enc_times))
    return {
        "value": flops_full / step / 1e12,
        "unit": "TFLOP/s",
        "cores": int(blas_threads),
        "os_cpu_count": os.cpu_count(),
        "blas_threads": int(blas_threads),
        "elementwise_threads": 1,
        "kind": "oracle",
        "sample": (f"the whole step of {M}x{N}x{K} (oracle encode of all {M} A rows, decode of "
                   f"A and of the {N} coded W rows, exact fp64 product), W coding excluded as "
                   f"on the GPU; {len(times)} repetitions, {sum(times):.1f} s measured; numpy "
                   f"elementwise on 1 thread, BLAS on {blas_threads}"),
        "seconds_per_step": step,
        "seconds_per_step_min": float(np.min(times)),
        "encode_A_seconds": enc,
        "encode_A_GBps": enc_bytes_of(cfg) / enc / 1e9,
    }


def enc_bytes_of(cfg):
    import workloads
    c = workloads.WORKLOADS[cfg]
    return algorithmic(c["M"], c["N"], c["K"], 4 if c["dtype"] == "f32" else 2)[0]


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1"}))
        sys.exit(2)

    if args.kv:
        kv_roofline(args)
        return
    if args.copy_bytes:
        copy_calibration(args)
        return
    if args.gemv:
        gemv_roofline(args)
        return
    if args.frontier:
        frontier(args)
        return

    import numpy as np
    import torch
    import workloads
    import paper_2502_09720_amd as nq

    cfg = args.workload
    c = workloads.WORKLOADS[cfg]
    M, N, K = c["M"], c["N"], c["K"]
    q = args.q or c["qs"][0]
    k = c["k"]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    sa, _, dta = workloads.operand(cfg, "A")
    sw, _, dtw = workloads.operand(cfg, "W")

    def up(store, dt):
        if dt == "bf16":
            return torch.from_numpy(store.view(np.int16)).to(dev).view(torch.bfloat16)
        return torch.from_numpy(store).to(dev)

    A0 = up(sa, dta)
    W = up(sw, dtw)
    del sa, sw
    in_bytes = A0.element_size()
    enc_bytes, mm_bytes, flops = algorithmic(M, N, K, in_bytes)
    nbuf = max(1, -(-512 * 2**20 // (M * K * in_bytes)) + 1)
    As = [A0] + [A0.clone() for _ in range(nbuf - 1)]

    # W is coded once (a weight) and kept in enough copies (at least 16, over 512 MiB in all)
    # that each step's read of the coded W comes from HBM, as for the layers of a model
    wc0 = nq.encode(W, q=q, k=k)
    del W
    nb, nbw = K // 8, (K // 8 + 15) // 16
    coded_w_bytes = N * nb * 4 + N * nbw * 4 + N * 4
    nw = max(16, -(-512 * 2**20 // coded_w_bytes))
    wcs = [wc0] + [wc0._replace(codes=wc0.codes.clone(), beta=wc0.beta.clone(),
                                scales=wc0.scales.clone()) for _ in range(nw - 1)]
    codes = torch.empty(M * nb, dtype=torch.int32, device=dev)
    beta = torch.empty(M * nbw, dtype=torch.int32, device=dev)
    scales = torch.empty(M, dtype=torch.float32, device=dev)
    C = torch.empty(M, N, dtype=torch.float32, device=dev)
    ws = torch.empty(max(1, nq.matmul_workspace_size(M, N, K)), dtype=torch.uint8, device=dev)

    # one step: nq_encode_matmul, the whole path in one call (encode A, whose encoder also
    # writes A's decoded tiles; decode of W; contraction)
    def step(i, ev=None):
        if ev is not None:
            ev[0].record()
        nq.encode_matmul(As[i % nbuf], wcs[i % nw], q=q, k=k, out=C,
                         coded_out=(codes, beta, scales), workspace=ws)
        if ev is not None:
            ev[1].record()

    for i in range(max(args.warmup, 1)):
        step(i)
    torch.cuda.synchronize()
    use_graph = args.graph
    if use_graph:
        # one captured graph of the step per activation buffer: a replay launches the
        # encoder, W's decode and the contraction with no host work between them
        graphs = []
        for b in range(nbuf):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                nq.encode_matmul(As[b], wcs[b % nw], q=q, k=k, out=C,
                                 coded_out=(codes, beta, scales), workspace=ws)
            graphs.append(g)
        torch.cuda.synchronize()

        def step(i, ev=None):
            if ev is not None:
                ev[0].record()
            graphs[i % nbuf].replay()   # buffer b pairs with W copy b % nw
            if ev is not None:
                ev[1].record()

        for i in range(args.warmup):
            step(i)
        torch.cuda.synchronize()
    # the timed region: K steps back to back (no event markers between them, which would
    # hold up the stream), then the same K steps again with an event pair around each one
    # for the per-step device time
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(i)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    sev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
    for i in range(args.steps):
        step(i, sev[i])
    torch.cuda.synchronize()
    step_t = stats([e[0].elapsed_time(e[1]) for e in sev])
    step_ev_ms = step_t["mean_ms"]

    # the same work as separate calls, with events between them on the kernels' stream:
    # nq_encode of A, then nq_matmul as its two stages (operand decode, contraction)
    def staged(i, ev):
        ev[0].record()
        ac = nq.encode(As[i % nbuf], q=q, k=k, out=(codes, beta, scales))
        ev[1].record()
        nq.matmul(ac, wcs[i % nw], out=C, workspace=ws, stages=nq.STAGE_DECODE)
        ev[2].record()
        nq.matmul(ac, wcs[i % nw], out=C, workspace=ws, stages=nq.STAGE_CONTRACT)
        ev[3].record()

    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    for i in range(args.warmup):
        staged(i, evs[i % args.steps])
    torch.cuda.synchronize()
    for i in range(args.steps):
        staged(i, evs[i])
    torch.cuda.synchronize()

    # the Hadamard rotation in front of the encoder (Sec. 5; not part of the step)
    rot = None
    try:
        Y = torch.empty(M, K, dtype=torch.float32, device=dev)
        for i in range(args.warmup):
            nq.rotate(As[i % nbuf], out=Y)
        torch.cuda.synchronize()
        er = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
        for i in range(args.steps):
            er[i][0].record()
            nq.rotate(As[i % nbuf], out=Y)
            er[i][1].record()
        torch.cuda.synchronize()
        rms = float(np.mean([e[0].elapsed_time(e[1]) for e in er]))
        rbytes = M * K * (in_bytes + 4)
        rot = {"ms": rms, "GBps": rbytes / (rms * 1e-3) / 1e9,
               "hbm_frac": rbytes / (rms * 1e-3) / 1e9 / HBM_PEAK_GBPS, "bytes": rbytes}

        def timed(fn):
            for i in range(args.warmup):
                fn(i)
            torch.cuda.synchronize()
            ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)]
                  for _ in range(args.steps)]
            for i in range(args.steps):
                ev[i][0].record()
                fn(i)
                ev[i][1].record()
            torch.cuda.synchronize()
            return float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))

        # rotation and coding of A in two passes (nq_rotate, then nq_encode of its fp32
        # rows), and in one (nq_rotate_encode: the rows rotated in LDS); then the whole step
        # on rotated operands (W coded once from its rotated rows)
        rot["rotate_then_encode_ms"] = timed(lambda i: (
            nq.rotate(As[i % nbuf], out=Y), nq.encode(Y, q=q, k=k, out=(codes, beta, scales))))
        del Y
        try:
            rot["rotate_encode_ms"] = timed(lambda i: nq.encode(
                As[i % nbuf], q=q, k=k, out=(codes, beta, scales), rotate=True))
            wc_rot = nq.encode(nq.rotate(up(workloads.operand(cfg, "W")[0], dtw)), q=q, k=k)
            rot["nq_encode_matmul_rotated_ms"] = timed(lambda i: nq.encode_matmul(
                As[i % nbuf], wc_rot, q=q, k=k, out=C, coded_out=(codes, beta, scales),
                workspace=ws, rotate=True))
            del wc_rot
        except nq.NQError:
            pass                              # a width the in-LDS rotation does not hold
    except nq.NQError:
        pass                                  # K not 2^k or 28 * 2^k

    # Opt-beta encoding of A (App. F; every beta tried, a strategy of the encoder that the
    # step does not use)
    eo = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
    for i in range(args.warmup):
        nq.encode(As[i % nbuf], q=q, k=k, out=(codes, beta, scales), strategy=nq.OPT_BETA)
    for i in range(args.steps):
        eo[i][0].record()
        nq.encode(As[i % nbuf], q=q, k=k, out=(codes, beta, scales), strategy=nq.OPT_BETA)
        eo[i][1].record()
    torch.cuda.synchronize()
    oms = float(np.mean([e[0].elapsed_time(e[1]) for e in eo]))
    opt = {"ms": oms, "GBps": enc_bytes / (oms * 1e-3) / 1e9}

    # the exact int8 contraction (a variant of the product, not part of the step)
    i8 = None
    if k * q <= 63:
        ev8 = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
        ac = nq.encode(As[0], q=q, k=k, out=(codes, beta, scales))
        for i in range(args.warmup):
            nq.matmul(ac, wcs[i % nw], out=C, workspace=ws, int8=True)
        for i in range(args.steps):
            ev8[i][0].record()
            nq.matmul(ac, wcs[i % nw], out=C, workspace=ws, stages=nq.STAGE_DECODE, int8=True)
            ev8[i][1].record()
            nq.matmul(ac, wcs[i % nw], out=C, workspace=ws, stages=nq.STAGE_CONTRACT, int8=True)
            ev8[i][2].record()
        torch.cuda.synchronize()
        d8 = float(np.mean([e[0].elapsed_time(e[1]) for e in ev8]))
        c8 = float(np.mean([e[1].elapsed_time(e[2]) for e in ev8]))
        i8 = {"decode_stage_ms": d8, "contract_stage_ms": c8,
              "contract_TOPs": flops / (c8 * 1e-3) / 1e12,
              "contract_int8_frac": flops / (c8 * 1e-3) / 1e12 / INT8_PEAK_TOPS,
              "matmul_TOPs": flops / ((d8 + c8) * 1e-3) / 1e12}

    enc_t = stats([e[0].elapsed_time(e[1]) for e in evs])
    dec_t = stats([e[1].elapsed_time(e[2]) for e in evs])
    con_t = stats([e[2].elapsed_time(e[3]) for e in evs])
    mm_t = stats([e[1].elapsed_time(e[3]) for e in evs])
    enc_ms, dec_ms, con_ms = enc_t["mean_ms"], dec_t["mean_ms"], con_t["mean_ms"]
    mm_ms = dec_ms + con_ms
    ms_per_step = wall * 1e3 / args.steps

    enc_gbps = enc_bytes / (enc_ms * 1e-3) / 1e9
    mm_tflops = flops / (mm_ms * 1e-3) / 1e12
    con_tflops = flops / (con_ms * 1e-3) / 1e12
    value = flops / (ms_per_step * 1e-3) / 1e12
    skinny = M <= 64
    if skinny:
        # decode-shaped product: the contraction kernel streams the coded W (HBM roofline)
        con_bytes = mm_bytes
        con_gbps = con_bytes / (con_ms * 1e-3) / 1e9
        roofline = {"kernel": "skinny_kernel (W decoded into 16x16x32 bf16 MFMA operands)",
                    "bound": "hbm", "achieved": con_gbps, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                    "frac": con_gbps / HBM_PEAK_GBPS, "traffic": None,
                    "per_launch": f"{con_bytes} algorithmic bytes (coded A, coded W, fp32 C)"}
    else:
        roofline = {"kernel": "gemm_kernel (bf16 MFMA contraction of the decoded tiles)",
                    "bound": "mfma", "achieved": con_tflops, "peak": BF16_PEAK_TFLOPS,
                    "unit": "TFLOP/s", "frac": con_tflops / BF16_PEAK_TFLOPS,
                    "traffic": gemm_traffic(cfg, q),
                    "per_launch": f"2*M*N*K = {flops:.4g} flops"}
    # the product from the codes as a whole (decode of both operands + contraction), the
    # quantity the decode-GEMM target is stated for
    decode_gemm = {"kernels": "operand decode + contraction (nq_matmul_stages)",
                   "bound": "mfma", "achieved": mm_tflops, "peak": BF16_PEAK_TFLOPS,
                   "unit": "TFLOP/s", "frac": mm_tflops / BF16_PEAK_TFLOPS,
                   "median_frac": flops / (mm_t["median_ms"] * 1e-3) / 1e12 / BF16_PEAK_TFLOPS,
                   "per_call": f"2*M*N*K = {flops:.4g} flops"}
    kv = None if args.no_kv else kv_measure(min(args.steps, 50), min(args.warmup, 20))

    out = {
        "metric": METRIC,
        "value": value,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": c["name"], "M": M, "N": N, "K": K, "q": q, "k": k,
            "A": f"{dta} {'Student-t(4)' if cfg == 3 else 'synthetic'}", "W": f"{dtw} coded once",
            "launch": "HIP graph replay of the step" if use_graph else "direct launches",
            "parallelism": "single GPU",
        },
        "components": {
            "nq_encode_matmul_ms": step_ev_ms,
            "nq_encode_matmul_stats": step_t,
            "nq_encode_ms": enc_ms,
            "nq_encode_stats": enc_t,
            "nq_encode_GBps": enc_gbps,
            "nq_encode_hbm_frac": enc_gbps / HBM_PEAK_GBPS,
            "nq_encode_bytes": enc_bytes,
            "nq_matmul_ms": mm_ms,
            "nq_matmul_stats": mm_t,
            "nq_matmul_decode_stage_ms": dec_ms,
            "nq_matmul_decode_stage_stats": dec_t,
            "nq_matmul_contract_stage_ms": con_ms,
            "nq_matmul_contract_stage_stats": con_t,
            "nq_matmul_TFLOPs": mm_tflops,
            "nq_matmul_mfma_frac": mm_tflops / BF16_PEAK_TFLOPS,
            "nq_matmul_bytes": mm_bytes,
            "a_rotation_buffers": nbuf,
            "w_coded_copies": nw,
            "kv_2e21x128_fp16": kv,
            "rate_bits_per_entry": float(np.log2(q) + np.log2(k) / 8),
            "nq_matmul_int8_variant": i8,
            "nq_rotate_A": rot,
            "nq_encode_A_opt_beta": opt,
        },
        "roofline": roofline,
        "decode_gemm": decode_gemm,
        "targets": {
            "encode_hbm_frac": enc_gbps / HBM_PEAK_GBPS,
            "decode_gemm_mfma_frac": mm_tflops / BF16_PEAK_TFLOPS,
            "kv_encode_hbm_frac": kv["nq_encode"]["hbm_frac"] if kv else None,
            "kv_decode_hbm_frac": kv["nq_decode"]["hbm_frac"] if kv else None,
            "stated": "encode >= 0.60 of 8 TB/s; decode-GEMM >= 0.50 of 2.5 PFLOP/s",
        },
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, q, k, flops)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
