"""Packed storage of a coded matrix: code words, beta-index words and row scales.

TEST INFRASTRUCTURE ONLY (see the package docstring).

App. E stores the eight codes of one block (each in [0, q), q <= 16) as the eight nibbles
of one 32-bit word, code i in bits 4i..4i+3, and each block's beta as an index into a
dictionary of four values, two bits per block.  The paper leaves the beta-index layout
open; this layout keeps, per row, ceil(blocks / 16) 32-bit words, with the index
(t - 1) of block j in bits 2 (j mod 16) of word j / 16.  Scales are one fp32 per row.
"""

import numpy as np


def codes_words(rows, cols):
    return rows * (cols // 8)


def beta_words(rows, cols):
    return rows * ((cols // 8 + 15) // 16)


def pack_codes(codes):
    """(rows, nb, 8) ints in [0, 16) -> (rows, nb) uint32."""
    c = np.asarray(codes, dtype=np.uint64)
    if np.any(c > 15):
        raise ValueError("codes must fit a nibble")
    shifts = (4 * np.arange(8)).astype(np.uint64)
    return (c << shifts).sum(axis=-1).astype(np.uint32)


def unpack_codes(words):
    w = np.asarray(words, dtype=np.uint32)[..., None]
    return ((w >> (4 * np.arange(8, dtype=np.uint32))) & 0xF).astype(np.int64)


def pack_beta(t):
    """(rows, nb) beta numbers t in [1, 4] -> (rows, ceil(nb / 16)) uint32 of 2-bit indices."""
    t = np.asarray(t, dtype=np.int64)
    if np.any((t < 1) | (t > 4)):
        raise ValueError("beta numbers must be in [1, 4]")
    rows, nb = t.shape
    nw = (nb + 15) // 16
    padded = np.zeros((rows, nw * 16), dtype=np.uint64)
    padded[:, :nb] = t - 1
    padded = padded.reshape(rows, nw, 16)
    shifts = (2 * np.arange(16)).astype(np.uint64)
    return (padded << shifts).sum(axis=-1).astype(np.uint32)


def unpack_beta(words, nb):
    w = np.asarray(words, dtype=np.uint32)
    rows, nw = w.shape
    idx = (w[:, :, None] >> (2 * np.arange(16, dtype=np.uint32))) & 3
    return idx.reshape(rows, nw * 16)[:, :nb].astype(np.int64) + 1
