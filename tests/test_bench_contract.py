"""CPU checks of bench.py's contract pieces: the one-GPU refusal, the algorithmic byte and
flop counts its roofline uses, and the rule that the counter-derived traffic is reported
only while the kernel source still matches the one the counters were taken on."""

import hashlib
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 2
    line = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in line["error"]


def test_algorithmic_counts_of_the_q_proj_shape():
    """2048 x 4096 x 4096 with bf16 input: A read once (16 MiB) plus its codes (4 bits per
    entry), beta words (2 bits per block) and fp32 scales; the product reads both coded
    operands and writes fp32 C; 2 M N K flops."""
    M, N, K = 2048, 4096, 4096
    enc, mm, flops = bench.algorithmic(M, N, K, 2)
    codes = lambda rows: rows * K // 2 + rows * (K // 128) * 4 + rows * 4  # noqa: E731
    assert enc == M * K * 2 + codes(M)
    assert mm == codes(M) + codes(N) + M * N * 4
    assert flops == 2.0 * M * N * K
    assert abs(enc / 1e6 - 21.2) < 0.1          # 16.8 MB in + 4.2 MB codes + beta + r
    assert abs(flops / 1e9 - 68.7) < 0.1


def test_gemm_traffic_follows_the_kernel_source():
    path = os.path.join(ROOT, "profiles", "gemm_kernel_workload3_traffic.md")
    if not os.path.exists(path):
        pytest.skip("no traffic summary")
    fields = {}
    for line in open(path):
        if line.startswith("- ") and ":" in line:
            key, val = line[2:].split(":", 1)
            fields[key.strip()] = val.strip().strip("`")
    src = os.path.join(ROOT, "paper_2502_09720_amd", "csrc", "nq_gemm.hip")
    fresh = hashlib.sha256(open(src, "rb").read()).hexdigest() == fields["kernel source sha256"]
    got = bench.gemm_traffic(3, 14)
    if fresh:
        assert got == float(fields["traffic bytes per launch"]) and got > 0
    else:
        assert got is None
    assert bench.gemm_traffic(3, 7) is None       # counters were taken at q = 14 only
