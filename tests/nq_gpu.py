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
