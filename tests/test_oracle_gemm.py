"""Pins of the oracle's dense product: numpy's fp64 matmul of the same fp32
inputs (a different library, rounded once the same way), every transposition,
alpha / beta, identity and rank-one closed forms."""
import numpy as np
import pytest


@pytest.mark.parametrize("ta", [False, True])
@pytest.mark.parametrize("tb", [False, True])
def test_matches_numpy_fp64(ref, ta, tb):
    rng = np.random.default_rng(10 * ta + tb)
    M, N, K = 37, 29, 53
    A = rng.standard_normal((K, M) if ta else (M, K)).astype(np.float32)
    B = rng.standard_normal((N, K) if tb else (K, N)).astype(np.float32)
    C = rng.standard_normal((M, N)).astype(np.float32)
    got = ref.gemm(A, B, ta, tb, alpha=0.75, beta=-1.5, C=C)
    a = A.astype(np.float64).T if ta else A.astype(np.float64)
    b = B.astype(np.float64).T if tb else B.astype(np.float64)
    want = (0.75 * (a @ b) - 1.5 * C.astype(np.float64)).astype(np.float32)
    assert np.max(np.abs(got.astype(np.float64) - want)) <= 2 * np.spacing(np.abs(want)).max()


def test_closed_forms(ref):
    rng = np.random.default_rng(3)
    X = rng.standard_normal((16, 16)).astype(np.float32)
    assert np.array_equal(ref.gemm(X, np.eye(16, dtype=np.float32)), X)
    assert np.array_equal(ref.gemm(np.eye(16, dtype=np.float32), X, tb=True), X.T.copy())
    u = np.arange(1, 9, dtype=np.float32)[:, None]
    assert np.array_equal(ref.gemm(u, u, tb=True), (u @ u.T).astype(np.float32))   # exact small integers
