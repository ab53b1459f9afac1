"""NestQuant coded GEMM on AMD Instinct MI355X (gfx950).

A thin Python layer over libnestquant.so (C ABI in include/nestquant.h): it marshals torch
device tensors and the current HIP stream into the C calls.  All arithmetic of the method
runs in the library's HIP kernels; there is no CPU fallback, and every call raises if the
library has not been built.
"""

from .binding import (  # noqa: F401
    CONTRACT_INT8,
    DECODER_FULL,
    DECODER_M,
    FIRST_BETA,
    OPT_BETA,
    ROTATE_A,
    STAGE_CONTRACT,
    STAGE_DECODE,
    Coded,
    NQError,
    beta_dp,
    beta_stats,
    decode,
    default_base,
    encode,
    encode_matmul,
    library,
    library_path,
    matmul,
    matmul_direct,
    matmul_workspace_size,
    nq_beta_words,
    nq_codes_words,
    rotate,
)
