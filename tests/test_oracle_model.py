"""Pins for the oracle's model step around the compressor: Eq. (11c) with the
node-summed tracker G, the optimisers of the experiments (Sec. VI: SGD as in
(11c), momentum SGD, Adam) and the dense warm-up (compression starts after a
number of dense iterations).

Every expected value here comes from a closed form or an invariant, on inputs
chosen so that binary32 evaluates it exactly (dyadic rationals), or from a
second, different route through the oracle (the identity compressor)."""
import numpy as np
import pytest

import oracle

F32 = np.float32


def _dyadic(rng, shape, lo=-64, hi=64, scale=2.0**-6):
    return (rng.integers(lo, hi, size=shape) * scale).astype(F32)


def test_sgd_is_eq_11c_in_closed_form():
    # G constant over T steps, lr and G/N dyadic: x_T = x_0 - T * lr * G / N.
    rng = np.random.default_rng(0)
    N, d, T, lr = 4, 1000, 7, 2.0**-3
    G = _dyadic(rng, d)
    x0 = _dyadic(rng, d)
    x = x0.copy()
    for t in range(T):
        oracle.optimizer_step("sgd", G, x, N=N, T=t + 1, lr=lr)
    want = x0.astype(np.float64) - T * lr * G.astype(np.float64) / N
    assert np.array_equal(x, want.astype(F32))
    assert np.array_equal(want.astype(F32).astype(np.float64), want)  # exact


def test_sgd_weight_decay_closed_form():
    # G = 0: x_T = x_0 * (1 - lr * wd)^T, exact for dyadic lr * wd.
    N, d, T, lr, wd = 2, 64, 5, 0.5, 0.25
    x0 = (np.arange(d) - 32).astype(F32)
    x = x0.copy()
    G = np.zeros(d, F32)
    for t in range(T):
        oracle.optimizer_step("sgd", G, x, N=N, T=t + 1, lr=lr, weight_decay=wd)
    assert np.array_equal(x, (x0 * (1 - lr * wd) ** T).astype(F32))


def test_msgd_heavy_ball_closed_form():
    # Constant direction dir = G / N, beta = 1/2, u_0 = 0:
    #   u_t = dir * (2 - 2^(1-t)),  x_T = x_0 - lr * sum_t u_t.
    rng = np.random.default_rng(1)
    N, d, T, lr, beta = 2, 500, 6, 2.0**-2, 0.5
    G = _dyadic(rng, d)
    x0 = _dyadic(rng, d)
    x, u = x0.copy(), np.zeros(d, F32)
    for t in range(T):
        oracle.optimizer_step("msgd", G, x, u, N=N, T=t + 1, lr=lr, momentum=beta)
    dir_ = G.astype(np.float64) / N
    u_want = dir_ * (2 - 2.0 ** (1 - T))
    x_want = x0 - lr * dir_ * sum(2 - 2.0 ** (1 - t) for t in range(1, T + 1))
    assert np.array_equal(u, u_want.astype(F32))
    assert np.array_equal(x, x_want.astype(F32))


def test_adam_moves_by_lr_times_sign_with_constant_direction():
    # beta1 = 1/2, beta2 = 3/4, eps = 0, constant dir = +-2^k: the bias
    # corrections give m_hat = dir and v_hat = dir^2 exactly at every step,
    # so each step moves x by exactly lr * sign(dir) (Kingma & Ba's Adam).
    N, d, T, lr = 4, 16, 5, 2.0**-4
    dir_ = np.array([(-1) ** j * 2.0 ** (j % 7 - 3) for j in range(d)], F32)
    G = (dir_ * N).astype(F32)
    x0 = np.linspace(-1, 1, d).astype(F32)
    x, m, v = x0.copy(), np.zeros(d, F32), np.zeros(d, F32)
    for t in range(T):
        oracle.optimizer_step("adam", G, x, m, v, N=N, T=t + 1, lr=lr, beta1=0.5, beta2=0.75,
                              eps=0.0)
        assert np.array_equal(x, (x0 - (t + 1) * lr * np.sign(dir_)).astype(F32)), t


def test_adam_first_step_is_normalised_direction():
    # Any beta1, beta2: after one step from m = v = 0, m_hat = dir and
    # v_hat = dir^2 up to rounding, so x moves by lr * dir / (|dir| + eps).
    rng = np.random.default_rng(2)
    N, d, lr, eps = 3, 4000, 1e-3, 1e-8
    G = rng.standard_normal(d).astype(F32)
    x0 = rng.standard_normal(d).astype(F32)
    x, m, v = x0.copy(), np.zeros(d, F32), np.zeros(d, F32)
    oracle.optimizer_step("adam", G, x, m, v, N=N, T=1, lr=lr, beta1=0.9, beta2=0.999, eps=eps)
    dir_ = G.astype(np.float64) / N
    want = x0 - lr * dir_ / (np.abs(dir_) + eps)
    assert np.max(np.abs(x - want)) <= 4 * np.finfo(F32).eps * np.max(np.abs(x0))
    assert np.allclose(m, 0.1 * dir_, rtol=1e-6) and np.allclose(v, 0.001 * dir_ ** 2, rtol=1e-5)


def test_adam_bias_correction_uses_the_step_count():
    # With a constant direction the corrected moments are dir and dir^2 at
    # every step count; a mistake in c1 or c2 (wrong T, or no correction)
    # moves x by a visibly different amount at a later step.
    N, d, lr = 1, 8, 2.0**-3
    dir_ = np.full(d, 0.25, F32)
    x, m, v = np.zeros(d, F32), np.zeros(d, F32), np.zeros(d, F32)
    for t in range(12):
        oracle.optimizer_step("adam", dir_.copy(), x, m, v, N=N, T=t + 1, lr=lr, beta1=0.9,
                              beta2=0.999, eps=0.0)
    assert np.allclose(x, -12 * lr, rtol=1e-5)


def test_dense_step_is_the_identity_compressor():
    # Second route: the compressor step with K >= m (every row kept) then
    # G += agg must give the same h, g, G bits as the dense step.
    rng = np.random.default_rng(3)
    N, d, n = 3, 64 * 37 + 5, 64
    grads = [rng.standard_normal((N, d)).astype(F32) for _ in range(3)]
    h1, g1, G1 = np.zeros((N, d), F32), np.zeros((N, d), F32), np.zeros(d, F32)
    h2, g2, G2 = h1.copy(), g1.copy(), G1.copy()
    for t, gr in enumerate(grads):
        oracle.dense_step(h1, g1, G1, gr, 0.1)
        out = oracle.step(h2, g2, gr, n=n, r=4, eta=0.1, seed=5, t=t, K=10**6)
        oracle.accumulate(G2, out["idx"], out["agg"], n=n)
    for a, b in ((h1, h2), (g1, g2), (G1, G2)):
        assert a.tobytes() == b.tobytes()


def test_dense_step_from_zero_sets_g_to_h_and_G_to_their_sum():
    rng = np.random.default_rng(4)
    N, d = 4, 999
    grad = _dyadic(rng, (N, d))
    h, g, G = np.zeros((N, d), F32), np.zeros((N, d), F32), np.zeros(d, F32)
    oracle.dense_step(h, g, G, grad, 0.5)
    assert np.array_equal(h, grad * F32(0.5))
    assert np.array_equal(g, h)
    assert np.array_equal(G, h.sum(axis=0))


def test_tracker_sum_invariant_over_compressed_steps():
    # G_t = sum_i g_t^(i): exact on dyadic inputs, through dense warm-up
    # steps and then compressed steps (payload added at the selected rows).
    rng = np.random.default_rng(5)
    N, d, n = 4, 32 * 50, 32
    h, g, G = np.zeros((N, d), F32), np.zeros((N, d), F32), np.zeros(d, F32)
    for t in range(8):
        grad = _dyadic(rng, (N, d))
        if t < 2:
            oracle.dense_step(h, g, G, grad, 0.5)
        else:
            out = oracle.step(h, g, grad, n=n, r=4, eta=0.5, seed=9, t=t, K=5)
            oracle.accumulate(G, out["idx"], out["agg"], n=n)
        assert np.array_equal(G, g.sum(axis=0)), t


def test_accumulate_tensors_places_rows_by_tensor():
    tensors = [(3, 4, 1), (1, 2, 1), (2, 3, 2)]
    d = 3 * 4 + 2 + 2 * 3
    G = np.zeros(d, F32)
    idx = np.array([2, 3, 4, 5], np.int32)  # row 2 of t0, row 0 of t1, rows 0, 1 of t2
    agg = np.arange(1, 4 + 2 + 6 + 1, dtype=F32)
    oracle.accumulate(G, idx, agg, tensors=tensors)
    want = np.zeros(d, F32)
    want[8:12] = agg[0:4]
    want[12:14] = agg[4:6]
    want[14:20] = agg[6:12]
    assert np.array_equal(G, want)
    with pytest.raises(oracle.OracleError):
        oracle.accumulate(G, np.array([0, 0, 4, 5], np.int32), agg, tensors=tensors)
