"""The byte-SIMD decoder (decode_word_b8: Alg. 2 with the Gosset oracle of Alg. 5, or
NestQuantM's of App. D) built for the host, its AMDGCN byte instructions replaced by C++
written from their ISA definitions (tests/host/nq_b8_host.cpp), against the oracle's
decoder: every code word for q <= 6, random words for every other q up to 16.  The GPU parity
tests run the same header on the device; this test covers every code word of small q,
including all the ties of Alg. 5, on the CPU.  CPU only."""

import ctypes
import os
import shutil
import subprocess

import numpy as np
import pytest

from conftest import ROOT
from oracle import voronoi

CSRC = os.path.join(ROOT, "paper_2502_09720_amd", "csrc")


@pytest.fixture(scope="module")
def host_decoder(tmp_path_factory):
    clang = "/opt/rocm/llvm/bin/clang++"
    if not os.path.exists(clang):
        clang = shutil.which("clang++")
    if clang is None:
        pytest.skip("needs clang++ (ext_vector_type and __builtin_elementwise_max)")
    so = str(tmp_path_factory.mktemp("b8") / "nq_b8_host.so")
    cmd = [clang, "-std=c++17", "-O2", "-shared", "-fPIC", "-Wall", "-I", CSRC,
           os.path.join(ROOT, "tests", "host", "nq_b8_host.cpp"), "-o", so]
    build = subprocess.run(cmd, capture_output=True, text=True)
    assert build.returncode == 0, build.stderr
    lib = ctypes.CDLL(so)
    lib.nq_b8_host_decode.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int,
                                      ctypes.c_int, ctypes.c_void_p]
    lib.nq_b8_host_decode.restype = None

    def decode(codes, q, decoder):
        codes = np.ascontiguousarray(codes, dtype=np.int64)
        words = np.zeros(len(codes), dtype=np.uint32)
        for i in range(8):                       # code i in bits 4i..4i+3 of the word
            words |= codes[:, i].astype(np.uint32) << np.uint32(4 * i)
        out = np.empty((len(codes), 8), dtype=np.int32)
        lib.nq_b8_host_decode(words.ctypes.data, len(codes), q, int(decoder == "m"),
                              out.ctypes.data)
        return out
    return decode


def all_codes(q):
    """Every c in {0..q-1}^8, one per row."""
    g = np.indices((q,) * 8, dtype=np.int64).reshape(8, -1).T
    return np.ascontiguousarray(g)


@pytest.mark.parametrize("decoder", ["full", "m"])
@pytest.mark.parametrize("q", [2, 3, 4, 5, 6])
def test_every_code_word(host_decoder, q, decoder):
    c = all_codes(q)
    got = host_decoder(c, q, decoder)
    want = voronoi.decode(c, q, decoder)
    bad = np.nonzero(np.any(got != want, axis=1))[0]
    assert bad.size == 0, (q, decoder, c[bad[:3]].tolist(), got[bad[:3]].tolist(),
                           want[bad[:3]].tolist())


@pytest.mark.parametrize("decoder", ["full", "m"])
@pytest.mark.parametrize("q", list(range(7, 17)))
def test_random_code_words(host_decoder, q, decoder):
    rng = np.random.default_rng(1000 + 17 * q + (decoder == "m"))
    c = rng.integers(0, q, size=(1 << 17, 8))
    # and the extremes: all codes 0, all q - 1, one code q - 1 among zeros and the converse
    eye = np.eye(8, dtype=np.int64)
    c = np.concatenate([c, np.zeros((1, 8), np.int64), np.full((1, 8), q - 1),
                        (q - 1) * eye, (q - 1) * (1 - eye)])
    got = host_decoder(c, q, decoder)
    want = voronoi.decode(c, q, decoder)
    bad = np.nonzero(np.any(got != want, axis=1))[0]
    assert bad.size == 0, (q, decoder, c[bad[:3]].tolist(), got[bad[:3]].tolist(),
                           want[bad[:3]].tolist())
