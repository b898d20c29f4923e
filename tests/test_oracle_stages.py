"""Pins for the oracle's per-stage arithmetic: momentum (Eq. (11a)), residual
sketch (Alg. 1), worker sum and row importance (Eq. (4)).

Each case fixes the expected value by hand, by a closed form, or by an exact
error bound against a binary64 library product, so that a dropped term, a
wrong sign or index, or a transposed operand fails.
"""
import numpy as np
import pytest

import oracle

F32 = np.float32


# --------------------------------------------------------------- momentum ---
def test_momentum_dyadic_by_hand():
    h = np.zeros((1, 3), F32)
    oracle.momentum(h, np.array([[2, 4, -8]], F32), 0.5)
    assert h.tolist() == [[1, 2, -4]]
    oracle.momentum(h, np.array([[0, 4, 8]], F32), 0.5)
    assert h.tolist() == [[0.5, 3, 2]]
    oracle.momentum(h, np.array([[4, 0, 0]], F32), 0.25)
    # 0.75*[0.5, 3, 2] + 0.25*[4, 0, 0]
    assert h.tolist() == [[1.375, 2.25, 1.5]]


def test_momentum_eta_one_copies_gradient():
    rng = np.random.default_rng(0)
    h = rng.standard_normal((3, 257)).astype(F32)
    grad = rng.standard_normal((3, 257)).astype(F32)
    oracle.momentum(h, grad, 1.0)
    assert np.array_equal(h, grad)


def test_momentum_constant_gradient_closed_form():
    # h_t = (1 - (1-eta)^t) c for a constant gradient c and h_0 = 0
    eta, c = 0.1, np.full((2, 64), 3.0, F32)
    h = np.zeros((2, 64), F32)
    for t in range(1, 41):
        oracle.momentum(h, c, eta)
        expect = (1.0 - (1.0 - eta) ** t) * 3.0
        np.testing.assert_allclose(h, expect, rtol=4e-6 * t)


def test_momentum_bf16_widening_is_exact():
    vals = np.array([1.5, -2.25, 3.0e-3, 1.0e20, -7.0], F32)
    bits = (vals.view(np.uint32) >> 16).astype(np.uint16)  # some bf16 bit patterns
    widened = (bits.astype(np.uint32) << 16).view(F32)
    h = np.zeros((1, 5), F32)
    oracle.momentum(h, bits[None, :], 1.0)
    assert np.array_equal(h[0], widened)


def test_momentum_rejects_bad_eta():
    h = np.zeros((1, 4), F32)
    for bad in (-0.1, 1.5, float("nan")):
        with pytest.raises(oracle.OracleError):
            oracle.momentum(h, np.zeros((1, 4), F32), bad)


# ----------------------------------------------------------------- sketch ---
def test_sketch_unit_columns_pick_row_entries():
    # V = [e_0, e_1, e_2] (n = 5, r = 3): S[i][p][k] = Delta[p*n + k] exactly.
    rng = np.random.default_rng(1)
    N, n, m = 3, 5, 7
    d = n * m
    h = rng.standard_normal((N, d)).astype(F32)
    g = rng.standard_normal((N, d)).astype(F32)
    V = np.zeros((n, 3), F32)
    V[0, 0] = V[1, 1] = V[2, 2] = 1.0
    S = oracle.sketch(h, g, V, n)
    delta = (h - g).reshape(N, m, n)
    assert np.array_equal(S, delta[:, :, :3])


def test_sketch_ones_gives_row_sums_and_ragged_tail():
    # d = 10, n = 4: rows {0..3}, {4..7}, {8, 9}; V = ones(r = 1) gives row sums.
    h = np.arange(1, 11, dtype=F32)[None, :]
    g = np.zeros_like(h)
    S = oracle.sketch(h, g, np.ones((4, 1), F32), 4)
    assert S[0, :, 0].tolist() == [1 + 2 + 3 + 4, 5 + 6 + 7 + 8, 9 + 10]


def test_sketch_is_sequential_in_j():
    # Delta = [2^24, 1, 1, -2^24], V = 1.  Ascending fmaf chain:
    # 2^24 -> fl(2^24 + 1) = 2^24 -> 2^24 -> 0.  The exact sum and the
    # descending order give 2; the pairwise order gives 1.
    h = np.array([[2.0 ** 24, 1.0, 1.0, -(2.0 ** 24)]], F32)
    S = oracle.sketch(h, np.zeros_like(h), np.ones((4, 1), F32), 4)
    assert S[0, 0, 0] == 0.0


def test_sketch_uses_residual_h_minus_g():
    h = np.array([[5.0, 1.0]], F32)
    g = np.array([[2.0, 4.0]], F32)
    S = oracle.sketch(h, g, np.array([[1.0], [10.0]], F32), 2)
    assert S[0, 0, 0] == (5 - 2) * 1 + (1 - 4) * 10


def test_sketch_within_error_bound_of_float64_product():
    # |fl(chain) - exact| <= gamma_n * sum_j |Delta_j V_jk|, gamma_n = n u / (1 - n u)
    rng = np.random.default_rng(2)
    N, n, m, r = 2, 384, 9, 4
    h = rng.standard_normal((N, n * m)).astype(F32)
    g = rng.standard_normal((N, n * m)).astype(F32)
    V = rng.standard_normal((n, r)).astype(F32)
    S = oracle.sketch(h, g, V, n).astype(np.float64)
    delta = (h - g).astype(np.float64).reshape(N, m, n)
    exact = delta @ V.astype(np.float64)
    u = 2.0 ** -24
    gamma = n * u / (1 - n * u)
    bound = gamma * (np.abs(delta) @ np.abs(V.astype(np.float64)))
    assert np.all(np.abs(S - exact) <= bound)
    # and the columns are not transposed: a swapped V fails the same bound
    swapped = delta @ V[:, ::-1].astype(np.float64)
    assert not np.all(np.abs(S - swapped) <= bound)


# ----------------------------------------------------- worker sum, Sigma ---
def test_worker_sum_is_sequential_in_i():
    # S over 4 workers = [2^24, 1, 1, -2^24]: ascending i gives 0
    # (descending gives 2, pairwise 1).
    S = np.array([2.0 ** 24, 1.0, 1.0, -(2.0 ** 24)], F32).reshape(4, 1, 1)
    assert oracle.worker_sum(S)[0, 0] == 0.0


def test_worker_sum_small_integers_exact():
    rng = np.random.default_rng(3)
    S = rng.integers(-50, 50, size=(5, 33, 4)).astype(F32)
    assert np.array_equal(oracle.worker_sum(S), S.sum(axis=0))


def test_importance_is_row_norm_squared():
    P = np.array([[1, 2, 3, 4], [0, 0, 0, 0], [-3, 0, 4, 0]], F32)
    assert oracle.importance(P).tolist() == [30.0, 0.0, 25.0]


def test_importance_nonnegative_and_bounded():
    rng = np.random.default_rng(4)
    P = rng.standard_normal((1000, 4)).astype(F32)
    s = oracle.importance(P).astype(np.float64)
    exact = (P.astype(np.float64) ** 2).sum(axis=1)
    assert np.all(s >= 0)
    assert np.all(np.abs(s - exact) <= 4 * 2.0 ** -24 * exact * 1.0001)
