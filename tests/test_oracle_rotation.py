"""Pins of the rotation oracle (Sec. 5): Hadamard matrices, orthogonality, the fp32 fast
transform against the exact product."""

import numpy as np
import pytest
import scipy.linalg

from oracle import rotation


@pytest.mark.parametrize("n", [1, 2, 8, 64, 1024])
def test_sylvester_matches_scipy(n):
    assert np.array_equal(rotation.sylvester(n), scipy.linalg.hadamard(n))


def test_paley28_is_hadamard():
    H = rotation.paley28()
    assert H.shape == (28, 28)
    assert set(np.unique(H)) == {-1, 1}
    assert np.array_equal(H @ H.T, 28 * np.eye(28, dtype=np.int64))


@pytest.mark.parametrize("n", [8, 128, 1024, 28 * 16])
def test_rotation_matrix_is_orthogonal(n):
    U = rotation.rotation_matrix(n)
    assert np.allclose(U @ U.T, np.eye(n), atol=1e-12)


@pytest.mark.parametrize("n", [8, 16, 128, 512, 2048, 28 * 8, 28 * 64, 14336])
def test_fast_rotation_matches_exact_product(n):
    """The fp32 fast transform is the exact product up to its roundings: each output is a
    sum of n terms of size |x|, so the error is below (log2 n + 28) * 2^-24 * sum |x|."""
    rng = np.random.default_rng(n)
    x = rng.standard_normal((6, n)).astype(np.float32)
    x[0, :] = 0.0
    x[1, n // 3] = 1e6                                # an outlier spreads over the row
    y = rotation.rotate_rows(x).astype(np.float64)
    # the exact product through the Kronecker structure: x (H1 kron H2) = H1^T X H2 per row
    m, p = rotation.split(n)
    H1 = np.ones((1, 1)) if m == 1 else rotation.paley28().astype(np.float64)
    H2 = scipy.linalg.hadamard(p).astype(np.float64)
    X = x.astype(np.float64).reshape(-1, m, p)
    exact = np.matmul(np.matmul(H1.T, X), H2).reshape(-1, n) / np.sqrt(n)
    bound = (np.log2(n) + 30) * 2.0 ** -24 * np.abs(x).astype(np.float64).sum(axis=1) / np.sqrt(n)
    assert np.all(np.abs(y - exact) <= bound[:, None] + 1e-30)
    assert np.all(y[0] == 0.0)


def test_rotation_preserves_norm_and_spreads_outliers():
    n = 4096
    x = np.zeros((1, n), np.float32)
    x[0, 17] = 3.0
    y = rotation.rotate_rows(x)
    assert np.allclose(np.abs(y), 3.0 / 64.0)         # one spike -> flat row, exactly
    rng = np.random.default_rng(1)
    x = rng.standard_normal((4, n)).astype(np.float32)
    y = rotation.rotate_rows(x)
    assert np.allclose(np.linalg.norm(y, axis=1), np.linalg.norm(x, axis=1), rtol=1e-5)


def test_rotation_twice_is_identity_for_symmetric_sylvester():
    """H_n / sqrt(n) is symmetric and orthogonal, so applying it twice returns the row."""
    rng = np.random.default_rng(2)
    x = rng.standard_normal((3, 256)).astype(np.float32)
    z = rotation.rotate_rows(rotation.rotate_rows(x))
    assert np.allclose(z, x, atol=1e-5)


def test_unsupported_sizes():
    assert rotation.split(24) is None
    assert rotation.split(11008) is None
    assert rotation.split(28672) == (28, 1024)


def test_conference14():
    """C of Paley's second construction: symmetric (q = 13 = 1 mod 4), zero diagonal,
    +-1 elsewhere and C C^T = 13 I, which makes C kron H_2 + I kron K_2 a Hadamard matrix."""
    C = rotation.conference14()
    assert np.array_equal(C, C.T)
    assert np.all(np.diag(C) == 0)
    assert set(np.unique(C[~np.eye(14, dtype=bool)])) == {-1, 1}
    assert np.array_equal(C @ C.T, 13 * np.eye(14, dtype=np.int64))


@pytest.mark.parametrize("p", [8, 64])
def test_mix_is_exact_on_integers(p):
    """Small integer rows keep every fp32 sum exact, so the fast transform followed by the
    H_28 sums must equal the integer product x (H_28 kron H_p) before the final scaling: any
    wrong sign or index in the transform or the mix shows."""
    n = 28 * p
    rng = np.random.default_rng(p)
    x = rng.integers(-8, 9, size=(5, n)).astype(np.float32)
    y = rotation.rotate_rows(x)
    H = np.kron(rotation.paley28(), scipy.linalg.hadamard(p)).astype(np.int64)
    S = x.astype(np.int64) @ H
    assert np.all(np.abs(S) < 2 ** 24)
    want = (S.astype(np.float32) * rotation.scale32(n)).astype(np.float32)
    assert np.array_equal(y, want)
