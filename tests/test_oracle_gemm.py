"""Pins of the oracle's INT8 product (the reference for decode-then-GEMM).

Checked against an independent int64 matrix product, hand-computed values, the
extreme operands the int8 ranges allow, and the int32 range guard.
"""
import numpy as np
import pytest


def test_hand_computed(oracle):
    a = np.array([[1, 2], [3, 4]], dtype=np.int8)
    b = np.array([[5, 6], [7, 8]], dtype=np.int8)
    # Y = A B^T: rows of A against rows of B
    assert oracle.gemm_i8_nt(a, b).tolist() == [[17, 23], [39, 53]]


@pytest.mark.parametrize("m,n,k", [(1, 1, 1), (7, 5, 3), (33, 17, 100), (64, 48, 513)])
def test_matches_int64_matmul(oracle, m, n, k):
    rng = np.random.default_rng([3, m, n, k])
    a = rng.integers(-128, 128, (m, k), dtype=np.int8)
    b = rng.integers(-128, 128, (n, k), dtype=np.int8)
    ref = a.astype(np.int64) @ b.astype(np.int64).T
    assert np.array_equal(oracle.gemm_i8_nt(a, b), ref)


def test_row_subset_equals_full_rows(oracle):
    rng = np.random.default_rng(9)
    a = rng.integers(-128, 128, (40, 64), dtype=np.int8)
    b = rng.integers(-128, 128, (24, 64), dtype=np.int8)
    rows = [39, 0, 17, 17]
    assert np.array_equal(oracle.gemm_i8_nt(a, b, rows=rows), oracle.gemm_i8_nt(a, b)[rows])


def test_extremes_and_int32_guard(oracle):
    k = 131072   # 16384 * 131072 = 2^31: one past the int32 range
    a = np.full((1, k - 1), -128, dtype=np.int8)
    assert oracle.gemm_i8_nt(a, a)[0, 0] == 16384 * (k - 1)
    big = np.full((1, k), -128, dtype=np.int8)
    with pytest.raises(RuntimeError):
        oracle.gemm_i8_nt(big, big)
