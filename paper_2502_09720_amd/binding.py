"""ctypes binding of libnestquant.so: argument marshalling only.

Device memory and streams come from torch; each function passes raw device pointers and
the current stream's handle to the matching C entry point and checks its status.
"""

import ctypes
import os
from typing import NamedTuple

PKG = os.path.dirname(os.path.abspath(__file__))
_LIB = None

NQ_OK, NQ_ERR_INVALID_ARG, NQ_ERR_UNSUPPORTED, NQ_ERR_HIP = 0, 1, 2, 3
NQ_F32, NQ_F16, NQ_BF16 = 0, 1, 2


class NQError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"{message} (status {status})")
        self.status = status


class _Params(ctypes.Structure):
    _fields_ = [("q", ctypes.c_int32), ("k", ctypes.c_int32), ("base", ctypes.c_double),
                ("decoder", ctypes.c_int32), ("strategy", ctypes.c_int32),
                ("mult", ctypes.c_int32 * 4)]


DECODER_FULL = 0   # Alg. 2 with the Gosset oracle of Alg. 5
DECODER_M = 1      # NestQuantM (App. D): parity fixes at the first coordinate
FIRST_BETA = 0     # App. F: the smallest beta that does not overload
OPT_BETA = 1       # App. F: the beta of least reconstruction error


def library_path():
    return os.environ.get("NESTQUANT_LIB") or os.path.join(PKG, "libnestquant.so")


def library():
    """Load libnestquant.so (raises if it has not been built)."""
    global _LIB
    if _LIB is None:
        path = library_path()
        if not os.path.exists(path):
            raise RuntimeError(
                f"{path} is missing: build it with `python -m paper_2502_09720_amd.build`")
        lib = ctypes.CDLL(path)
        vp, i64, u32p, f32p = ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p
        pp = ctypes.POINTER(_Params)
        lib.nq_encode.argtypes = [pp, vp, ctypes.c_int, i64, i64, i64, u32p, u32p, f32p, vp]
        lib.nq_rotate_encode.argtypes = lib.nq_encode.argtypes
        lib.nq_rotate_encode.restype = ctypes.c_int
        lib.nq_decode.argtypes = [pp, u32p, u32p, f32p, i64, i64, vp, ctypes.c_int, i64, vp]
        lib.nq_matmul.argtypes = [pp, u32p, u32p, f32p, i64, pp, u32p, u32p, f32p, i64, i64,
                                  f32p, i64, vp]
        lib.nq_matmul_ex.argtypes = [pp, u32p, u32p, f32p, i64, pp, u32p, u32p, f32p, i64, i64,
                                     f32p, i64, vp, i64, vp]
        lib.nq_matmul_stages.argtypes = [ctypes.c_int32, pp, u32p, u32p, f32p, i64, pp, u32p,
                                         u32p, f32p, i64, i64, f32p, i64, vp, i64, vp]
        lib.nq_encode_matmul.argtypes = [ctypes.c_int32, pp, vp, ctypes.c_int, i64, i64, i64,
                                         u32p, u32p, f32p, pp, u32p, u32p, f32p, i64, f32p, i64,
                                         vp, i64, vp]
        lib.nq_encode_matmul.restype = ctypes.c_int
        lib.nq_rotate.argtypes = [vp, ctypes.c_int, i64, i64, i64, f32p, i64, vp]
        lib.nq_rotate.restype = ctypes.c_int
        i32 = ctypes.c_int32
        lib.nq_beta_stats.argtypes = [i32, i32, vp, i64, ctypes.POINTER(ctypes.c_double), i32,
                                      vp, vp, vp]
        lib.nq_beta_stats.restype = ctypes.c_int
        lib.nq_beta_dp.argtypes = [vp, vp, i64, i32, i32, vp, vp, vp, i64, vp]
        lib.nq_beta_dp.restype = ctypes.c_int
        lib.nq_beta_dp_workspace_size.argtypes = [i64, i32]
        lib.nq_beta_dp_workspace_size.restype = i64
        lib.nq_matmul_workspace_size.argtypes = [i64, i64, i64]
        lib.nq_matmul_workspace_size.restype = i64
        for f in ("nq_encode", "nq_decode", "nq_matmul", "nq_matmul_ex", "nq_matmul_stages"):
            getattr(lib, f).restype = ctypes.c_int
        lib.nq_codes_words.argtypes = [i64, i64]
        lib.nq_codes_words.restype = i64
        lib.nq_beta_words.argtypes = [i64, i64]
        lib.nq_beta_words.restype = i64
        lib.nq_status_string.argtypes = [ctypes.c_int]
        lib.nq_status_string.restype = ctypes.c_char_p
        lib.nq_last_error.argtypes = []
        lib.nq_last_error.restype = ctypes.c_char_p
        lib.nq_version.argtypes = []
        lib.nq_version.restype = ctypes.c_int32
        _LIB = lib
    return _LIB


def _check(status):
    if status != NQ_OK:
        lib = library()
        raise NQError(status, lib.nq_last_error().decode() or lib.nq_status_string(status).decode())


def default_base(q, k):
    """beta_t = t * base with the k betas uniform on [0, 10] / q."""
    return 10.0 / (k * q)


def _params(q, k, base, decoder=DECODER_FULL, strategy=FIRST_BETA, mult=None):
    m = [0, 0, 0, 0]
    if mult is not None:
        m[:len(mult)] = [int(v) for v in mult]
    return _Params(int(q), int(k), float(default_base(q, k) if base is None else base),
                   int(decoder), int(strategy), (ctypes.c_int32 * 4)(*m))


def _stream(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _dtype_code(dt):
    import torch
    return {torch.float32: NQ_F32, torch.float16: NQ_F16, torch.bfloat16: NQ_BF16}[dt]


def nq_codes_words(rows, cols):
    return library().nq_codes_words(rows, cols)


def nq_beta_words(rows, cols):
    return library().nq_beta_words(rows, cols)


class Coded(NamedTuple):
    """A coded matrix: uint32 code words (stored in an int32 tensor), uint32 beta words,
    fp32 row scales, and the quantizer parameters (mult: the integer multiples of base that
    make the betas, None for 1..k)."""
    codes: "object"
    beta: "object"
    scales: "object"
    rows: int
    cols: int
    q: int
    k: int
    base: float
    decoder: int = DECODER_FULL
    mult: "object" = None


def encode(x, q=14, k=4, base=None, stream=None, out=None, decoder=DECODER_FULL,
           strategy=FIRST_BETA, mult=None, rotate=False):
    """nq_encode on a 2-D cuda tensor (fp32 / fp16 / bf16, unit stride along rows).
    ``decoder`` is the decoder the code is defined with (DECODER_FULL or DECODER_M);
    ``strategy`` picks the beta of each block (FIRST_BETA or OPT_BETA); ``mult`` gives the
    betas as integer multiples of base (k increasing integers in [1, 64]; None: 1..k).
    ``rotate``: the rows are Hadamard-rotated (as ``rotate``) before they are coded: in one
    pass (nq_rotate_encode) where the library supports it (First-beta; cols in 3584, 4096,
    7168, 8192, 14336, 16384), else as nq_rotate into a temporary fp32 matrix followed by
    nq_encode (same results)."""
    import torch
    if x.dim() != 2 or x.stride(1) != 1 or not x.is_cuda:
        raise ValueError("x must be a 2-D cuda tensor with unit column stride")
    rows, cols = x.shape
    lib = library()
    nw, bw = lib.nq_codes_words(rows, cols), lib.nq_beta_words(rows, cols)
    if nw < 0:
        raise ValueError("cols must be a positive multiple of 8")
    if out is None:
        codes = torch.empty(nw, dtype=torch.int32, device=x.device)
        beta = torch.empty(bw, dtype=torch.int32, device=x.device)
        scales = torch.empty(rows, dtype=torch.float32, device=x.device)
    else:
        codes, beta, scales = out
    p = _params(q, k, base, decoder, strategy, mult)

    def call(fn, src):
        return fn(ctypes.byref(p), ctypes.c_void_p(src.data_ptr()), _dtype_code(src.dtype), rows,
                  cols, src.stride(0), ctypes.c_void_p(codes.data_ptr()),
                  ctypes.c_void_p(beta.data_ptr()), ctypes.c_void_p(scales.data_ptr()),
                  _stream(stream))
    st = call(lib.nq_rotate_encode if rotate else lib.nq_encode, x)
    if rotate and st == NQ_ERR_UNSUPPORTED:
        st = call(lib.nq_encode, _rotated(x, stream))                     # two passes
    _check(st)
    return Coded(codes, beta, scales, rows, cols, int(q), int(k), p.base, int(decoder),
                 None if mult is None else tuple(int(v) for v in mult))


def decode(coded, out_dtype=None, stream=None, out=None):
    """nq_decode: the reconstruction r * beta_t * p as a rows x cols tensor."""
    import torch
    dt = torch.float32 if out_dtype is None else out_dtype
    if out is None:
        out = torch.empty(coded.rows, coded.cols, dtype=dt, device=coded.codes.device)
    p = _params(coded.q, coded.k, coded.base, coded.decoder, mult=coded.mult)
    lib = library()
    _check(lib.nq_decode(ctypes.byref(p), ctypes.c_void_p(coded.codes.data_ptr()),
                         ctypes.c_void_p(coded.beta.data_ptr()),
                         ctypes.c_void_p(coded.scales.data_ptr()), coded.rows, coded.cols,
                         ctypes.c_void_p(out.data_ptr()), _dtype_code(out.dtype), out.stride(0),
                         _stream(stream)))
    return out


STAGE_DECODE = 1
STAGE_CONTRACT = 2
CONTRACT_INT8 = 4
ROTATE_A = 8


def matmul(a, w, stream=None, out=None, workspace=None, stages=STAGE_DECODE | STAGE_CONTRACT,
           int8=False):
    """nq_matmul: C = A_hat W_hat^T (fp32, M x N) from two coded operands.

    The decode-once workspace is taken from torch's allocator unless given.  ``stages``
    selects part of the call (nq_matmul_stages): STAGE_DECODE fills the workspace,
    STAGE_CONTRACT computes C from it; both (the default) is the whole product.  ``int8``
    contracts exact int8 tiles on int8 matrix cores (needs k * q <= 63)."""
    import torch
    if a.cols != w.cols:
        raise ValueError("K mismatch")
    if out is None:
        out = torch.empty(a.rows, w.rows, dtype=torch.float32, device=a.codes.device)
    pa = _params(a.q, a.k, a.base, a.decoder, mult=a.mult)
    pw = _params(w.q, w.k, w.base, w.decoder, mult=w.mult)
    lib = library()
    need = lib.nq_matmul_workspace_size(a.rows, w.rows, a.cols)
    if need < 0:
        raise ValueError("invalid matmul shape")
    whole = stages == STAGE_DECODE | STAGE_CONTRACT
    if need > 0 and (workspace is None or workspace.numel() * workspace.element_size() < need):
        if not whole:
            raise ValueError("a staged matmul needs a workspace of matmul_workspace_size bytes")
        workspace = torch.empty(need, dtype=torch.uint8, device=a.codes.device)
        if stream is not None:
            workspace.record_stream(stream)       # freed on return, in use on `stream`
    ws_ptr = workspace.data_ptr() if need > 0 else 0
    args = (ctypes.byref(pa), ctypes.c_void_p(a.codes.data_ptr()),
            ctypes.c_void_p(a.beta.data_ptr()), ctypes.c_void_p(a.scales.data_ptr()), a.rows,
            ctypes.byref(pw), ctypes.c_void_p(w.codes.data_ptr()),
            ctypes.c_void_p(w.beta.data_ptr()), ctypes.c_void_p(w.scales.data_ptr()), w.rows,
            a.cols, ctypes.c_void_p(out.data_ptr()), out.stride(0), ctypes.c_void_p(ws_ptr),
            need, _stream(stream))
    if whole and not int8:
        _check(lib.nq_matmul_ex(*args))
    else:
        _check(lib.nq_matmul_stages(stages | (CONTRACT_INT8 if int8 else 0), *args))
    return out


def matmul_direct(a, w, stream=None, out=None):
    """nq_matmul: C = A_hat W_hat^T with no workspace (each workgroup decodes the code words
    of its own rows into on-chip memory); the same product as ``matmul``."""
    import torch
    if a.cols != w.cols:
        raise ValueError("K mismatch")
    if out is None:
        out = torch.empty(a.rows, w.rows, dtype=torch.float32, device=a.codes.device)
    pa = _params(a.q, a.k, a.base, a.decoder, mult=a.mult)
    pw = _params(w.q, w.k, w.base, w.decoder, mult=w.mult)
    _check(library().nq_matmul(
        ctypes.byref(pa), ctypes.c_void_p(a.codes.data_ptr()), ctypes.c_void_p(a.beta.data_ptr()),
        ctypes.c_void_p(a.scales.data_ptr()), a.rows, ctypes.byref(pw),
        ctypes.c_void_p(w.codes.data_ptr()), ctypes.c_void_p(w.beta.data_ptr()),
        ctypes.c_void_p(w.scales.data_ptr()), w.rows, a.cols, ctypes.c_void_p(out.data_ptr()),
        out.stride(0), _stream(stream)))
    return out


def encode_matmul(x, w, q=14, k=4, base=None, decoder=DECODER_FULL, strategy=FIRST_BETA,
                  mult=None, stream=None, out=None, coded_out=None, workspace=None,
                  int8=False, rotate=False):
    """nq_encode_matmul: codes the activation x (2-D cuda tensor, as ``encode``) and returns
    (its Coded operand, C = A_hat W_hat^T) from one call, the encoder writing A's decoded
    tiles straight into the product's workspace.  The same results as ``encode`` then
    ``matmul``.  ``rotate``: x's rows are Hadamard-rotated before they are coded (w must hold
    the codes of rotated weight rows): NQ_ROTATE_A where the library supports it (as for
    ``encode``), else nq_rotate into a temporary fp32 matrix first (same results)."""
    import torch
    if x.dim() != 2 or x.stride(1) != 1 or not x.is_cuda:
        raise ValueError("x must be a 2-D cuda tensor with unit column stride")
    M, K = x.shape
    if K != w.cols:
        raise ValueError("K mismatch")
    lib = library()
    if coded_out is None:
        codes = torch.empty(max(lib.nq_codes_words(M, K), 0), dtype=torch.int32, device=x.device)
        beta = torch.empty(max(lib.nq_beta_words(M, K), 0), dtype=torch.int32, device=x.device)
        scales = torch.empty(M, dtype=torch.float32, device=x.device)
    else:
        codes, beta, scales = coded_out
    if out is None:
        out = torch.empty(M, w.rows, dtype=torch.float32, device=x.device)
    need = lib.nq_matmul_workspace_size(M, w.rows, K)
    if need < 0:
        raise ValueError("invalid matmul shape")
    if need > 0 and (workspace is None or workspace.numel() * workspace.element_size() < need):
        workspace = torch.empty(need, dtype=torch.uint8, device=x.device)
        if stream is not None:
            workspace.record_stream(stream)       # freed on return, in use on `stream`
    pa = _params(q, k, base, decoder, strategy, mult)
    pw = _params(w.q, w.k, w.base, w.decoder, mult=w.mult)

    def call(flags, src):
        return lib.nq_encode_matmul(
            flags, ctypes.byref(pa), ctypes.c_void_p(src.data_ptr()), _dtype_code(src.dtype), M,
            K, src.stride(0), ctypes.c_void_p(codes.data_ptr()),
            ctypes.c_void_p(beta.data_ptr()), ctypes.c_void_p(scales.data_ptr()),
            ctypes.byref(pw), ctypes.c_void_p(w.codes.data_ptr()),
            ctypes.c_void_p(w.beta.data_ptr()), ctypes.c_void_p(w.scales.data_ptr()), w.rows,
            ctypes.c_void_p(out.data_ptr()), out.stride(0),
            ctypes.c_void_p(workspace.data_ptr() if need > 0 else 0), need, _stream(stream))
    flags = CONTRACT_INT8 if int8 else 0
    st = call(flags | (ROTATE_A if rotate else 0), x)
    if rotate and st == NQ_ERR_UNSUPPORTED:
        st = call(flags, _rotated(x, stream))                                # two passes
    _check(st)
    a = Coded(codes, beta, scales, M, K, int(q), int(k), pa.base, int(decoder),
              None if mult is None else tuple(int(v) for v in mult))
    return a, out


def rotate(x, out=None, stream=None):
    """nq_rotate: y = x U in fp32 for every row of a 2-D cuda tensor (Sec. 5 Hadamard
    rotation; cols = 2^k or 28 * 2^k, at most 32768)."""
    import torch
    if x.dim() != 2 or x.stride(1) != 1 or not x.is_cuda:
        raise ValueError("x must be a 2-D cuda tensor with unit column stride")
    rows, cols = x.shape
    if out is None:
        out = torch.empty(rows, cols, dtype=torch.float32, device=x.device)
    _check(library().nq_rotate(ctypes.c_void_p(x.data_ptr()), _dtype_code(x.dtype), rows, cols,
                               x.stride(0), ctypes.c_void_p(out.data_ptr()), out.stride(0),
                               _stream(stream)))
    return out


def _rotated(x, stream):
    """nq_rotate of x into a new fp32 matrix (the two-pass form of the rotating calls).  The
    temporary is freed when the caller returns, so it is marked as in use on `stream` until
    the work queued there is done."""
    y = rotate(x, stream=stream)
    if stream is not None:
        y.record_stream(stream)
    return y


def matmul_workspace_size(M, N, K):
    return library().nq_matmul_workspace_size(M, N, K)


def beta_stats(v, betas, q, decoder=DECODER_FULL, stream=None):
    """nq_beta_stats: for sample 8-vectors v (n x 8 fp32 cuda tensor) and the increasing
    candidate betas (a sequence of at most 64 floats), the squared coding error mse (n x m
    fp64) and the overload flags (n x m uint8) of every sample at every beta."""
    import torch
    if v.dim() != 2 or v.shape[1] != 8 or v.dtype != torch.float32 or not v.is_contiguous():
        raise ValueError("v must be a contiguous n x 8 float32 cuda tensor")
    n, m = v.shape[0], len(betas)
    mse = torch.empty(n, m, dtype=torch.float64, device=v.device)
    over = torch.empty(n, m, dtype=torch.uint8, device=v.device)
    b = (ctypes.c_double * m)(*[float(x) for x in betas])
    _check(library().nq_beta_stats(int(q), int(decoder), ctypes.c_void_p(v.data_ptr()), n, b,
                                   m, ctypes.c_void_p(mse.data_ptr()),
                                   ctypes.c_void_p(over.data_ptr()), _stream(stream)))
    return mse, over


def beta_dp(mse, over, k, stream=None, workspace=None):
    """nq_beta_dp (Alg. 6): the k grid indices (int32 cuda tensor, increasing; -1 if every
    beta overloads) minimizing the First-beta error, and that error (fp64 cuda scalar).  The
    scratch memory (nq_beta_dp_workspace_size bytes) comes from torch's allocator unless
    given."""
    import torch
    n, m = mse.shape
    lib = library()
    chosen = torch.empty(k, dtype=torch.int32, device=mse.device)
    loss = torch.empty((), dtype=torch.float64, device=mse.device)
    need = lib.nq_beta_dp_workspace_size(n, m)
    if need < 0:
        raise ValueError("invalid beta_dp shape")
    if workspace is None or workspace.numel() * workspace.element_size() < need:
        workspace = torch.empty(max(need, 8), dtype=torch.uint8, device=mse.device)
        if stream is not None:
            workspace.record_stream(stream)       # freed on return, in use on `stream`
    _check(lib.nq_beta_dp(ctypes.c_void_p(mse.data_ptr()), ctypes.c_void_p(over.data_ptr()),
                          n, m, int(k), ctypes.c_void_p(chosen.data_ptr()),
                          ctypes.c_void_p(loss.data_ptr()), ctypes.c_void_p(workspace.data_ptr()),
                          workspace.numel() * workspace.element_size(), _stream(stream)))
    return chosen, loss
