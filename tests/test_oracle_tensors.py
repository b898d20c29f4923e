"""Pins for the oracle's per-tensor mode (Sec. VI: each tensor compressed in
its own 2-D view with its own K; 1-D tensors kept whole)."""
import math

import numpy as np
import pytest

import oracle

F32 = np.float32
# (rows, cols, K): a conv kernel 8 x (3*3*3) as out x in*kh*kw, a 1-D bias kept
# whole as one row, a 2-D weight and another 1-D vector.
LAYOUT = [(8, 27, 2), (1, 8, 1), (16, 12, 3), (1, 16, 1)]


def _d(layout):
    return sum(r * c for r, c, _ in layout)


def test_identity_when_every_tensor_is_kept_whole():
    # K_b = rows_b everywhere: the packed payload is the whole residual, in
    # order, summed over workers in ascending order.
    layout = [(r, c, r) for r, c, _ in LAYOUT]
    d, N = _d(layout), 3
    rng = np.random.default_rng(1)
    h = rng.standard_normal((N, d)).astype(F32)
    g = rng.standard_normal((N, d)).astype(F32)
    grad = rng.standard_normal((N, d)).astype(F32)
    g0 = g.copy()
    out = oracle.step_tensors(h, g, grad, layout, r=4, eta=0.3, seed=5, t=2)
    delta = h - g0
    acc = delta[0].copy()
    for i in range(1, N):
        acc = (acc + delta[i]).astype(F32)
    assert out["idx"].tolist() == list(range(sum(r for r, _, _ in layout)))
    assert np.array_equal(out["agg"], acc)
    assert np.array_equal(g, (g0 + delta).astype(F32))


def test_selection_is_per_tensor_and_rows_are_tensor_rows():
    d, N = _d(LAYOUT), 2
    rng = np.random.default_rng(2)
    grad = rng.standard_normal((N, d)).astype(F32)
    h = np.zeros((N, d), F32)
    g = np.zeros((N, d), F32)
    out = oracle.step_tensors(h, g, grad, LAYOUT, r=4, eta=1.0, seed=9, t=0, want_sigma=True)
    idx, sig = out["idx"].tolist(), out["sigma"]
    row0, q = 0, 0
    for rows, cols, K in LAYOUT:
        k = min(K, rows)
        mine = idx[q:q + k]
        want = sorted(sorted(range(row0, row0 + rows), key=lambda p: (-sig[p], p))[:k])
        assert mine == want
        row0 += rows
        q += k
    # packed payload: each selected row carries its tensor's width
    assert out["agg"].size == sum(min(K, r) * c for r, c, K in LAYOUT)


def test_sigma_uses_the_projection_of_each_width():
    # Sigma of a row = || sum_i Delta_i(row) V_w ||^2 with V_w = projection(seed, t, w)
    d, N = _d(LAYOUT), 2
    rng = np.random.default_rng(3)
    grad = rng.integers(-3, 4, size=(N, d)).astype(F32)
    h = np.zeros((N, d), F32)
    g = np.zeros((N, d), F32)
    out = oracle.step_tensors(h, g, grad, LAYOUT, r=4, eta=1.0, seed=11, t=4, want_sigma=True)
    off, row0 = 0, 0
    for rows, cols, _ in LAYOUT:
        V = oracle.projection(11, 4, cols, 4).astype(np.float64)
        x = grad.astype(np.float64).sum(axis=0)[off:off + rows * cols].reshape(rows, cols)
        exact = ((x @ V) ** 2).sum(axis=1)
        bound = 8 * cols * 2.0 ** -24 * ((np.abs(x) @ np.abs(V)) ** 2).sum(axis=1) + 1e-30
        assert np.all(np.abs(out["sigma"][row0:row0 + rows] - exact) <= bound)
        off += rows * cols
        row0 += rows


def test_matches_bucketed_single_view_when_widths_agree():
    # All tensors of width 16: the per-tensor step is the bucketed step with
    # the tensors as buckets (same V, same rows, same packed payload).
    layout = [(5, 16, 2), (9, 16, 4), (3, 16, 3)]
    d, N = _d(layout), 3
    rng = np.random.default_rng(4)
    grads = [rng.standard_normal((N, d)).astype(F32) for _ in range(3)]
    h1, g1 = np.zeros((N, d), F32), np.zeros((N, d), F32)
    h2, g2 = np.zeros((N, d), F32), np.zeros((N, d), F32)
    begin = [0, 5, 14, 17]
    ks = [2, 4, 3]
    for t, gr in enumerate(grads):
        a = oracle.step_tensors(h1, g1, gr, layout, r=4, eta=0.2, seed=3, t=t)
        b = oracle.step(h2, g2, gr, n=16, r=4, eta=0.2, seed=3, t=t, buckets=(begin, ks))
        assert a["idx"].tobytes() == b["idx"].tobytes()
        assert a["agg"].tobytes() == b["agg"].ravel().tobytes()
    assert h1.tobytes() == h2.tobytes() and g1.tobytes() == g2.tobytes()


def test_contraction_per_tensor_in_expectation():
    # Prop. 2 per tensor: mean over seeds of ||C(x_b) - x_b||^2 / ||x_b||^2 <= 1 - K_b/m_b
    layout = [(24, 32, 4), (12, 96, 2)]
    d, N = _d(layout), 4
    rng = np.random.default_rng(5)
    scale = np.concatenate([np.repeat(np.geomspace(0.1, 3, r)[rng.permutation(r)], c)
                            for r, c, _ in layout]).astype(F32)
    grad = (rng.standard_normal((N, d)) * scale).astype(F32)
    x = grad.astype(np.float64).mean(axis=0)
    ratios = {0: [], 1: []}
    for seed in range(400):
        h = np.zeros((N, d), F32)
        g = np.zeros((N, d), F32)
        out = oracle.step_tensors(h, g, grad, layout, r=4, eta=1.0, seed=seed, t=0)
        off, q, a = 0, 0, 0
        for b, (rows, cols, K) in enumerate(layout):
            xb = x[off:off + rows * cols].reshape(rows, cols)
            C = np.zeros_like(xb)
            row0 = sum(lr for lr, _, _ in layout[:b])
            for j in range(K):
                C[out["idx"][q + j] - row0] = out["agg"][a + j * cols:a + (j + 1) * cols] / N
            ratios[b].append(np.sum((C - xb) ** 2) / np.sum(xb ** 2))
            off += rows * cols
            q += K
            a += K * cols
    for b, (rows, cols, K) in enumerate(layout):
        r_ = np.array(ratios[b])
        assert r_.mean() <= 1 - K / rows + 3 * r_.std(ddof=1) / math.sqrt(len(r_))
        assert r_.mean() < 0.7 * (1 - K / rows)


def test_rejects_bad_layouts():
    h = np.zeros((1, 16), F32)
    with pytest.raises(oracle.OracleError):
        oracle.step_tensors(h, h.copy(), h.copy(), [(2, 8, -1)], r=4, eta=0.1, seed=0, t=0)
    with pytest.raises(ValueError):
        oracle.step_tensors(h, h.copy(), h.copy(), [(2, 7, 1)], r=4, eta=0.1, seed=0, t=0)
