"""Pins of the CPU oracle to facts fixed outside of it.

Each pin takes a loaded oracle library and raises AssertionError when the oracle
disagrees with an independent fact: a library routine on the special case it
covers, exact integer arithmetic on brute-forced tiny inputs, closed-form
invariants of the masked product, or the hand-worked fixture under
``tests/golden/``. ``test_oracle.py`` runs them against the real oracle, and
against builds with a planted mistake, which at least one pin must catch.
"""
from __future__ import annotations

import itertools
import os

import numpy as np

import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def f16(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64).astype(np.float16)).view(np.uint16)


def pin_f16_decode_all_patterns(lib):
    """All 65,536 binary16 patterns decode like numpy's float16 -> float64 cast."""
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    got = oracle.f16_to_f64(bits, lib=lib)
    ref = bits.view(np.float16).astype(np.float64)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    # signed zeros keep their sign
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan]))


def _py_masked(Wi, Mi, Xi):
    """Exact Python-integer masked product, token-major output [N][M]."""
    M, K = len(Wi), len(Wi[0])
    N = len(Xi)
    return [[sum(Wi[m][k] * Xi[n][k] for k in range(K) if Mi[m][k]) for m in range(M)]
            for n in range(N)]


def pin_bruteforce_2x4_all_masks(lib):
    """Every one of the 256 masks of a 2 x 4 W, small-integer W and X, vs exact integers."""
    rng = np.random.default_rng(7)
    Wi = rng.integers(-3, 4, size=(2, 4))
    Xi = rng.integers(-3, 4, size=(3, 4))
    Wb, Xb = f16(Wi), f16(Xi)
    for code in range(256):
        mask = np.array([[(code >> (4 * r + c)) & 1 for c in range(4)] for r in range(2)], dtype=np.uint8)
        Y, A = oracle.masked_gemm(Wb, mask, Xb, lib=lib)
        exp = np.array(_py_masked(Wi.tolist(), mask.tolist(), Xi.tolist()), dtype=np.float64)
        expA = np.array(_py_masked(np.abs(Wi).tolist(), mask.tolist(), np.abs(Xi).tolist()), dtype=np.float64)
        assert np.array_equal(Y, exp), code
        assert np.array_equal(A, expA), code


def pin_bruteforce_4x4_all_masks(lib):
    """All 65,536 masks of a 4 x 4 W at once (stacked as row blocks), vs exact int64 arithmetic."""
    rng = np.random.default_rng(11)
    Wi = rng.integers(-3, 4, size=(4, 4))
    Xi = rng.integers(-3, 4, size=(2, 4))
    codes = np.arange(1 << 16, dtype=np.int64)
    bits = ((codes[:, None] >> np.arange(16)[None, :]) & 1).astype(np.uint8)  # (65536, 16)
    mask = bits.reshape(-1, 4)  # row block c holds the 4 rows of mask code c
    Wall = np.tile(Wi, (1 << 16, 1))
    Y, _ = oracle.masked_gemm(f16(Wall), mask, f16(Xi), lib=lib)
    exp = (Wall * mask.astype(np.int64)) @ Xi.T  # exact integers, (M, N)
    assert np.array_equal(Y, exp.T.astype(np.float64))


def pin_dense_mask_is_gemm(lib):
    """All-ones mask: equals numpy's float64 matrix product of the fp16 inputs."""
    rng = np.random.default_rng(3)
    W = f16(rng.normal(0, 0.02, size=(37, 300)))
    X = f16(rng.normal(0, 1, size=(5, 300)))
    Y, A = oracle.masked_gemm(W, np.ones(W.shape, np.uint8), X, lib=lib)
    ref = W.view(np.float16).astype(np.float64) @ X.view(np.float16).astype(np.float64).T
    assert np.allclose(Y, ref.T, rtol=1e-12, atol=1e-12 * np.abs(A).max())
    refA = np.abs(W.view(np.float16).astype(np.float64)) @ np.abs(X.view(np.float16).astype(np.float64)).T
    assert np.allclose(A, refA.T, rtol=1e-12, atol=0)


def pin_zero_mask(lib):
    rng = np.random.default_rng(5)
    W = f16(rng.normal(0, 1, size=(9, 33)))
    X = f16(rng.normal(0, 1, size=(4, 33)))
    Y, A = oracle.masked_gemm(W, np.zeros(W.shape, np.uint8), X, lib=lib)
    assert np.all(Y == 0) and np.all(A == 0)


def pin_identity_columns(lib):
    """X = [e_j1 ... e_jN] returns the kept columns j1..jN of W exactly."""
    rng = np.random.default_rng(13)
    M, K = 23, 40
    W = f16(rng.normal(0, 0.02, size=(M, K)))
    mask = (rng.random((M, K)) < 0.5).astype(np.uint8)
    cols = np.array([0, 3, 17, 39, 20])
    Xd = np.zeros((cols.size, K))
    Xd[np.arange(cols.size), cols] = 1.0
    Y, _ = oracle.masked_gemm(W, mask, f16(Xd), lib=lib)
    Wm = np.where(mask != 0, W.view(np.float16).astype(np.float64), 0.0)
    assert np.array_equal(Y, Wm[:, cols].T)


def pin_additive_over_disjoint_masks(lib):
    rng = np.random.default_rng(17)
    M, K, N = 31, 64, 6
    W = f16(rng.normal(0, 0.02, size=(M, K)))
    X = f16(rng.normal(0, 1, size=(N, K)))
    u = rng.random((M, K))
    m1 = (u < 0.3).astype(np.uint8)
    m2 = ((u >= 0.3) & (u < 0.7)).astype(np.uint8)
    Y1, A1 = oracle.masked_gemm(W, m1, X, lib=lib)
    Y2, A2 = oracle.masked_gemm(W, m2, X, lib=lib)
    Y12, A12 = oracle.masked_gemm(W, m1 | m2, X, lib=lib)
    assert np.allclose(Y1 + Y2, Y12, rtol=0, atol=1e-13 * max(1.0, A12.max()))
    assert np.allclose(A1 + A2, A12, rtol=1e-13, atol=0)


def pin_row_permutation(lib):
    rng = np.random.default_rng(19)
    M, K, N = 29, 50, 3
    W = f16(rng.normal(0, 0.02, size=(M, K)))
    X = f16(rng.normal(0, 1, size=(N, K)))
    mask = (rng.random((M, K)) < 0.4).astype(np.uint8)
    p = rng.permutation(M)
    Y, _ = oracle.masked_gemm(W, mask, X, lib=lib)
    Yp, _ = oracle.masked_gemm(W[p], mask[p], X, lib=lib)
    assert np.array_equal(Yp, Y[:, p])
    # explicit row selection matches the full product
    Ys, _ = oracle.masked_gemm(W, mask, X, rows=p[:7], lib=lib)
    assert np.array_equal(Ys, Y[:, p[:7]])


def pin_power_of_two_scaling(lib):
    rng = np.random.default_rng(23)
    M, K, N = 17, 45, 4
    W = f16(rng.normal(0, 0.02, size=(M, K)))
    Xv = rng.normal(0, 1, size=(N, K)).astype(np.float16).astype(np.float64)
    mask = (rng.random((M, K)) < 0.5).astype(np.uint8)
    Y, _ = oracle.masked_gemm(W, mask, f16(Xv), lib=lib)
    Y8, _ = oracle.masked_gemm(W, mask, f16(Xv * 8.0), lib=lib)
    assert np.array_equal(Y8, 8.0 * Y)


def pin_abs_bound(lib):
    """|Y| <= A everywhere, with equality when all kept W and all X are nonnegative."""
    rng = np.random.default_rng(29)
    M, K, N = 21, 70, 5
    W = f16(rng.normal(0, 0.02, size=(M, K)))
    X = f16(rng.normal(0, 1, size=(N, K)))
    mask = (rng.random((M, K)) < 0.5).astype(np.uint8)
    Y, A = oracle.masked_gemm(W, mask, X, lib=lib)
    assert np.all(np.abs(Y) <= A * (1 + 1e-12))
    Wp = f16(np.abs(W.view(np.float16).astype(np.float64)))
    Xp = f16(np.abs(X.view(np.float16).astype(np.float64)))
    Y2, A2 = oracle.masked_gemm(Wp, mask, Xp, lib=lib)
    assert np.allclose(Y2, A2, rtol=1e-14, atol=0)


def pin_special_values(lib):
    """Subnormals kept exactly; Inf/NaN follow IEEE arithmetic; masked entries vanish entirely."""
    sub = 2.0 ** -24  # smallest fp16 subnormal
    X = f16([[1.0, 2.0, 1.0, np.inf]])
    W = f16([[sub, 3 * sub, -sub, 1.0],
             [np.inf, 1.0, 0.0, 0.0],
             [np.nan, 1.0, 0.0, 0.0],
             [np.nan, 1.0, 0.0, 0.0],
             [0.0, 1.0, 0.0, 0.0],
             [-0.0, -0.0, 0.0, 0.0]])
    mask = np.array([[1, 1, 1, 0],
                     [1, 1, 1, 0],
                     [0, 1, 1, 0],
                     [1, 1, 0, 0],
                     [0, 1, 0, 1],
                     [1, 1, 1, 0]], np.uint8)
    Y, A = oracle.masked_gemm(W, mask, X, lib=lib)
    y = Y[0]
    assert y[0] == 6 * sub and A[0, 0] == 8 * sub  # subnormals; masked 1 * Inf ignored
    assert np.isposinf(y[1])  # kept Inf weight
    assert y[2] == 2.0  # masked NaN weight ignored
    assert np.isnan(y[3])  # kept NaN weight
    assert np.isnan(y[4])  # kept exact zero times Inf
    assert y[5] == 0.0  # signed zeros


def pin_golden_hand_example(lib):
    path = os.path.join(GOLDEN, "spmm_hand_example.txt")
    vals: dict = {}
    for line in open(path):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        key, *rest = line.split()
        vals.setdefault(key, []).append([float(v) for v in rest])
    M, K, N = int(vals["M"][0][0]), int(vals["K"][0][0]), int(vals["N"][0][0])
    W = f16(np.array(vals["W"]))
    mask = np.array(vals["mask"], dtype=np.uint8)
    X = f16(np.array(vals["X"]))
    assert W.shape == (M, K) and X.shape == (N, K)
    Y, A = oracle.masked_gemm(W, mask, X, lib=lib)
    assert np.array_equal(Y, np.array(vals["Y"]).T)
    assert np.array_equal(A, np.array(vals["A"]).T)


def pin_masked_bits(lib):
    rng = np.random.default_rng(31)
    W = rng.integers(0, 1 << 16, size=(13, 27)).astype(np.uint16)
    mask = (rng.random(W.shape) < 0.5).astype(np.uint8) * rng.integers(1, 256, size=W.shape).astype(np.uint8)
    got = oracle.masked_bits(W, mask, lib=lib)
    for m, k in itertools.product(range(13), range(27)):
        assert got[m, k] == (W[m, k] if mask[m, k] else 0)


ALL_PINS = [
    pin_f16_decode_all_patterns,
    pin_bruteforce_2x4_all_masks,
    pin_bruteforce_4x4_all_masks,
    pin_dense_mask_is_gemm,
    pin_zero_mask,
    pin_identity_columns,
    pin_additive_over_disjoint_masks,
    pin_row_permutation,
    pin_power_of_two_scaling,
    pin_abs_bound,
    pin_special_values,
    pin_golden_hand_example,
    pin_masked_bits,
]
