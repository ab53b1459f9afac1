"""Helpers for the GPU parity tests: host<->device transfer and oracle wrappers.

The oracle side always works from the host arrays produced by ``workloads``; nothing it
consumes comes from the GPU path.
"""

import numpy as np

from oracle import layout, nestquant


def torch_mod():
    import torch
    return torch


def to_device(store, dtype):
    """Host storage (uint16 bf16 bits / float16 / float32) -> cuda tensor of that dtype."""
    torch = torch_mod()
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(store).view(np.int16)).cuda()
        return t.view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(store)).cuda()


def u32(t, shape=None):
    a = t.cpu().numpy().view(np.uint32)
    return a if shape is None else a.reshape(shape)


def oracle_encode(x32, q, k, base=None, decoder="full", strategy="first", mult=None):
    """Packed oracle codes (rows, nb), beta words (rows, nbw) and scales (rows,)."""
    codes, t, r = nestquant.quantize_rows(x32, q, k, base, strategy=strategy, decoder=decoder,
                                          mult=mult)
    return layout.pack_codes(codes), layout.pack_beta(t), r


def upload_coded(codes_w, beta_w, scales, rows, cols, q, k, base, decoder=0, mult=None):
    """Oracle-packed arrays -> a device Coded operand (decoder: 0 full, 1 NestQuantM; mult:
    the betas' multiples of base, None for 1..k)."""
    torch = torch_mod()
    from paper_2502_09720_amd import Coded
    c = torch.from_numpy(np.ascontiguousarray(codes_w).reshape(-1).view(np.int32)).cuda()
    b = torch.from_numpy(np.ascontiguousarray(beta_w).reshape(-1).view(np.int32)).cuda()
    s = torch.from_numpy(np.ascontiguousarray(scales, dtype=np.float32)).cuda()
    return Coded(c, b, s, rows, cols, q, k, base, decoder,
                 None if mult is None else tuple(int(v) for v in mult))


def first_mismatch(a, b):
    idx = np.argwhere(a != b)
    if len(idx) == 0:
        return None
    i = tuple(idx[0])
    return f"{len(idx)} mismatches, first at {i}: got {a[i]!r} want {b[i]!r}"


def ulp_in(dtype, v):
    """Spacing of the target dtype at |v| (fp64 v)."""
    v = np.abs(np.asarray(v, np.float64))
    if dtype == "f32":
        return np.spacing(v.astype(np.float32)).astype(np.float64)
    if dtype == "f16":
        return np.spacing(v.astype(np.float16)).astype(np.float64)
    # bf16: 8 significant bits
    e = np.floor(np.log2(np.maximum(v, 2.0 ** -126)))
    return 2.0 ** (e - 7)


def decoded_to_f64(t, dtype):
    torch = torch_mod()
    if dtype == "bf16":
        return t.view(torch.int16).cpu().numpy().view(np.uint16).astype(np.uint32).__lshift__(16) \
            .view(np.float32).astype(np.float64)
    return t.cpu().numpy().astype(np.float64)


# ----------------------------------------------------------------------------------------
# The oracle over many rows at once.  Coding is row-local, so the rows are split into chunks
# that worker processes code independently (the oracle itself, unchanged).  Workers are
# started with "spawn": fresh interpreters that never touch the GPU.
# ----------------------------------------------------------------------------------------

def _oracle_chunk(x32, q, k, base, decoder, mult, tiles):
    codes, t, r = nestquant.quantize_rows(x32, q, k, base, decoder=decoder, mult=mult)
    T = nestquant.integer_tiles(codes, t, q, decoder, mult).astype(np.int16) if tiles else None
    return layout.pack_codes(codes), layout.pack_beta(t), r, T


def oracle_encode_many(x32, q, k, base=None, decoder="full", mult=None, tiles=True,
                       workers=None):
    """Packed codes (rows, nb), beta words (rows, nbw), scales (rows,) and, with ``tiles``,
    the integer tiles m X2 as int16 (rows, cols): the oracle's quantize_rows on row chunks in
    worker processes (at most 16: the host share of one GPU)."""
    import concurrent.futures
    import multiprocessing
    import os
    rows = x32.shape[0]
    if workers is None:
        workers = max(1, min(16, os.cpu_count() or 1))
    chunk = max(64, -(-rows // (4 * workers)))
    parts = [(x32[i:i + chunk], q, k, base, decoder, mult, tiles) for i in range(0, rows, chunk)]
    import sys
    # spawned workers re-import the main module: only possible when it is a file
    spawnable = getattr(sys.modules.get("__main__"), "__file__", None) is not None
    if workers == 1 or len(parts) == 1 or not spawnable:
        out = [_oracle_chunk(*p) for p in parts]
    else:
        ctx = multiprocessing.get_context("spawn")
        progress = os.environ.get("NQ_TEST_PROGRESS") == "1"
        out = []
        with concurrent.futures.ProcessPoolExecutor(max_workers=min(workers, len(parts)),
                                                    mp_context=ctx) as ex:
            for i, o in enumerate(ex.map(_oracle_chunk, *zip(*parts), timeout=900)):
                out.append(o)
                if progress and (i + 1) % 16 == 0:
                    print(f"  oracle: {i + 1}/{len(parts)} chunks of {rows} rows", flush=True)
    codes = np.concatenate([o[0] for o in out])
    beta = np.concatenate([o[1] for o in out])
    r = np.concatenate([o[2] for o in out])
    T = np.concatenate([o[3] for o in out]) if tiles else None
    return codes, beta, r, T
