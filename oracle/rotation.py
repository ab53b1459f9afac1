"""Online Hadamard rotation of rows before quantization (Sec. 5, "LLM quantization").

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper rotates every weight-activation pair by an orthogonal U (A W^T = (A U)(W U)^T):

* n = 2^k: U = H_n / sqrt(n) with H_n the Sylvester Hadamard matrix;
* n = 2^k m with a Hadamard matrix H_1 of small order m: U = (H_1 kron H_2) / sqrt(n), H_2
  the Sylvester matrix of order 2^k.  The build supports m = 28 (Llama-3's 14336 = 28 * 512
  and 28672 = 28 * 1024), with H_28 from Paley's second construction at q = 13.

Readings (the paper fixes neither the arithmetic nor the order-28 matrix, whose table says
only "hardcoded Hadamard"):

* y = x U is computed in fp32 as a fast Walsh-Hadamard transform: for h = 1, 2, 4, ...,
  2^(k-1), every pair (i, i + h) with i & h = 0 becomes (a + b, a - b), one fp32 rounding
  per sum; the row is read as X[i, j] = x[i 2^k + j], i < m, and the transform runs along j.
* For m = 28, output segment a of the H_1 factor is the plain matrix product written out:
  the sum over i = 0..27, in increasing i, of H_28[i, a] X_i (X_i the i-th length-2^k
  segment after the transform), starting from H_28[0, a] X_0, fp32 with one rounding per
  addition (each term is an exact +-X_i).
* Finally every entry is multiplied once by fl32(1 / sqrt(n)) (fl64 square root and
  division first; a power of two when n is a power of four).
* H_28 (Paley II, q = 13 = 1 mod 4): with chi the quadratic character mod 13 and the
  symmetric 14 x 14 conference matrix C = [[0, 1^T], [1, Q]], Q[i, j] = chi(j - i),
  H_28 = C kron [[1, 1], [1, -1]] + I_14 kron [[1, -1], [-1, -1]].
"""

import numpy as np


def sylvester(n):
    """The Sylvester Hadamard matrix of order n (a power of two) by the doubling rule."""
    H = np.ones((1, 1), dtype=np.int64)
    while H.shape[0] < n:
        H = np.block([[H, H], [H, -H]])
    if H.shape[0] != n:
        raise ValueError("n must be a power of two")
    return H


def conference14():
    """The symmetric 14 x 14 conference matrix C = [[0, 1^T], [1, Q]] of Paley's second
    construction at q = 13: Q[i, j] = chi(j - i), chi the quadratic character mod 13."""
    q = 13
    residues = {(x * x) % q for x in range(1, q)}
    chi = np.array([0] + [1 if a in residues else -1 for a in range(1, q)], dtype=np.int64)
    Q = np.array([[chi[(j - i) % q] for j in range(q)] for i in range(q)], dtype=np.int64)
    C = np.zeros((q + 1, q + 1), dtype=np.int64)
    C[0, 1:] = 1
    C[1:, 0] = 1
    C[1:, 1:] = Q
    return C


def paley28():
    """A Hadamard matrix of order 28 by Paley's second construction with q = 13."""
    C = conference14()
    return (np.kron(C, np.array([[1, 1], [1, -1]]))
            + np.kron(np.eye(14, dtype=np.int64), np.array([[1, -1], [-1, -1]])))


def split(n):
    """n -> (m, 2^k) with m in {1, 28}, or None if the rotation is not supported."""
    for m in (1, 28):
        if n % m == 0:
            p = n // m
            if p >= 1 and p & (p - 1) == 0 and (m == 1 or p >= 1):
                return m, p
    return None


def rotation_matrix(n):
    """U = (H_1 kron H_2) / sqrt(n) in fp64 (H_1 = [1] for n a power of two)."""
    m, p = split(n)
    H1 = np.ones((1, 1), dtype=np.int64) if m == 1 else paley28()
    return np.kron(H1, sylvester(p)).astype(np.float64) / np.sqrt(n)


def scale32(n):
    """fl32(1 / sqrt(n)) from fp64 square root and division."""
    return np.float32(1.0 / np.sqrt(np.float64(n)))


def rotate_rows(x32):
    """y = x U for every row of x (rows, n), in the fp32 operation order of the docstring."""
    x = np.asarray(x32, dtype=np.float32)
    rows, n = x.shape
    sp = split(n)
    if sp is None:
        raise ValueError(f"no rotation for n = {n}")
    m, p = sp
    X = x.reshape(rows, m, p).copy()
    h = 1
    while h < p:
        Y = X.reshape(rows, m, p // (2 * h), 2, h)
        a = Y[:, :, :, 0, :].copy()
        b = Y[:, :, :, 1, :].copy()
        Y[:, :, :, 0, :] = a + b                       # fp32 adds: one rounding each
        Y[:, :, :, 1, :] = a - b
        X = Y.reshape(rows, m, p)
        h *= 2
    if m == 28:
        H1 = paley28()
        out = np.empty_like(X)
        for a in range(28):
            acc = X[:, 0, :] * np.float32(H1[0, a])                # exact +-X_0
            for i in range(1, 28):
                acc = acc + X[:, i, :] * np.float32(H1[i, a])     # one rounding per sum
            out[:, a, :] = acc
        X = out
    return (X.reshape(rows, n) * scale32(n)).astype(np.float32)
