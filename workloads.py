"""Seeded synthetic operands shaped like the Llama-3 layers the paper quantizes.

This module only draws and rounds random numbers; it holds none of the method's
arithmetic.  The tests, the oracle-timing leg of the benchmark and the GPU runs all take
their inputs from here, so every side sees identical bytes.

The paper evaluates on Llama-3-8B / 70B weights and WikiText2 activations (Sec. 5), which
are not available; these draws stand in for them with the same shapes:

  workload 1  A 64x512, W 256x512, fp32 iid N(0,1)                               (small case)
  workload 2  A 16x4096 bf16 N(0,1); W 14336x4096 bf16 N(0,0.02^2)               (decode-shaped)
  workload 3  A 2048x4096 bf16 Student-t(4); W 4096x4096 bf16 N(0,0.02^2)        (8B q_proj)
  workload 4  A 4096x14336 bf16 N(0,1) with 143 columns (1%) scaled by 20;
         W 4096x14336 bf16 N(0,0.02^2)                                      (8B down_proj)
  workload 5  A 2048x8192 bf16 N(0,1); W 28672x8192 bf16 N(0,0.015^2);
         X 2^21 x 128 fp16 N(0,1) (2^28 entries, KV-cache-like rows)         (70B MLP)

Recipe: each operand has its own stream ``numpy.random.default_rng([w, j])``, w the
workload number and j = 0 for A, 1 for W, 2 for X; values are drawn in float64 (in row chunks, so a row range can be
generated alone), scaled, and rounded once to the stored dtype (round to nearest even).
"""

import numpy as np

CHUNK_ROWS = 1 << 14

WORKLOADS = {
    1: dict(name="coded GEMM 64x256x512 fp32 N(0,1)", M=64, N=256, K=512, dtype="f32",
            qs=(14,), k=4),
    2: dict(name="decode-shaped linear 16x14336x4096 bf16", M=16, N=14336, K=4096, dtype="bf16",
            qs=(14,), k=4),
    3: dict(name="Llama-3-8B q_proj prefill 2048x4096x4096 bf16 (A Student-t4)", M=2048, N=4096,
            K=4096, dtype="bf16", qs=(14,), k=4),
    4: dict(name="Llama-3-8B down_proj prefill 4096x4096x14336 bf16 (1% x20 outlier columns)",
            M=4096, N=4096, K=14336, dtype="bf16", qs=(14, 7), k=4),
    5: dict(name="70B-scale MLP 2048x28672x8192 bf16 + 2^28 fp16 KV rows", M=2048, N=28672,
            K=8192, dtype="bf16", qs=(14,), k=4, X_rows=1 << 21, X_cols=128),
}


# ----------------------------------------------------------------------------------------
# single rounding from float64
# ----------------------------------------------------------------------------------------

def f64_to_bf16_bits(x):
    """Round float64 to bfloat16 (nearest, ties to even) once; returns uint16 bit patterns.

    float64 -> float32 with round-to-odd, then float32 -> bfloat16 with round-to-nearest-even:
    the odd intermediate keeps the sticky bit, so the result equals one direct rounding.
    """
    x = np.asarray(x, dtype=np.float64)
    f = x.astype(np.float32)
    over = np.abs(f.astype(np.float64)) > np.abs(x)
    f = np.where(over, np.nextafter(f, np.float32(0)), f)              # toward zero
    bits = f.view(np.uint32).copy()
    inexact = f.astype(np.float64) != x
    bits |= inexact.astype(np.uint32)                                   # round to odd
    finite = np.isfinite(f)
    lsb = (bits >> 16) & 1
    rounded = ((bits.astype(np.uint64) + 0x7FFF + lsb) >> 16).astype(np.uint16)
    return np.where(finite, rounded, (bits >> 16).astype(np.uint16))


def bf16_bits_to_f32(b):
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def round_to(x64, dtype):
    """Return (storage array, exact float32 view) for the stored dtype."""
    if dtype == "bf16":
        bits = f64_to_bf16_bits(x64)
        return bits, bf16_bits_to_f32(bits)
    if dtype == "f16":
        h = np.asarray(x64, dtype=np.float64).astype(np.float16)
        return h, h.astype(np.float32)
    if dtype == "f32":
        f = np.asarray(x64, dtype=np.float64).astype(np.float32)
        return f, f
    raise ValueError(dtype)


# ----------------------------------------------------------------------------------------
# operands
# ----------------------------------------------------------------------------------------

def _draw(cfg, which, rows, cols, row_range=None):
    """float64 draws for rows [lo, hi) of operand `which` ("A", "W" or "X")."""
    lo, hi = (0, rows) if row_range is None else row_range
    j = {"A": 0, "W": 1, "X": 2}[which]
    rng = np.random.default_rng([cfg, j])
    outlier_cols = None
    if cfg == 4 and which == "A":
        outlier_cols = np.sort(rng.choice(cols, size=cols // 100, replace=False))
    out = np.empty((hi - lo, cols), dtype=np.float64)
    for c0 in range(0, rows, CHUNK_ROWS):
        c1 = min(rows, c0 + CHUNK_ROWS)
        if c1 <= lo:
            # skip a whole chunk without drawing it: chunks use their own sub-streams
            continue
        if c0 >= hi:
            break
        sub = np.random.default_rng([cfg, j, c0 // CHUNK_ROWS])
        if cfg == 3 and which == "A":
            blk = sub.standard_t(4.0, size=(c1 - c0, cols))
        else:
            blk = sub.standard_normal(size=(c1 - c0, cols))
        a, b = max(lo, c0), min(hi, c1)
        out[a - lo:b - lo] = blk[a - c0:b - c0]
    if which == "W":
        out *= 0.015 if cfg == 5 else 0.02
    if outlier_cols is not None:
        out[:, outlier_cols] *= 20.0
    return out


def operand(cfg, which, row_range=None):
    """Operand `which` of config `cfg`: (storage, fp32 view, dtype).

    storage is uint16 bf16 bits, float16 or float32; the fp32 view holds the same values.
    row_range=(lo, hi) returns only those rows, identical to the full draw's rows.
    """
    c = WORKLOADS[cfg]
    if which == "A":
        rows, cols, dt = c["M"], c["K"], c["dtype"]
    elif which == "W":
        rows, cols, dt = c["N"], c["K"], c["dtype"]
    elif which == "X":
        rows, cols, dt = c["X_rows"], c["X_cols"], "f16"
    else:
        raise ValueError(which)
    x64 = _draw(cfg, which, rows, cols, row_range)
    store, f32 = round_to(x64, dt)
    return store, f32, dt


def outlier_columns(cfg=4):
    c = WORKLOADS[cfg]
    rng = np.random.default_rng([cfg, 0])
    return np.sort(rng.choice(c["K"], size=c["K"] // 100, replace=False))


def random_rows(seed, rows, cols, dtype="f32", scale=1.0, dist="normal"):
    """Small seeded matrices for parity and edge-case tests."""
    rng = np.random.default_rng(seed)
    if dist == "normal":
        x = rng.standard_normal((rows, cols))
    elif dist == "t4":
        x = rng.standard_t(4.0, size=(rows, cols))
    elif dist == "uniform":
        x = rng.uniform(-1.0, 1.0, size=(rows, cols))
    else:
        raise ValueError(dist)
    return round_to(x * scale, dtype)
