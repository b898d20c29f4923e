"""Pins for the oracle's comparison compressors of Table I inside the EF21M
step: Rand-K (shared random rows, summed payload) and Top-K (each node's own
rows by exact row norm, All-Gather payload).  Expected values come from the
published SplitMix64 outputs, Prop. 1's worked example, brute force in
binary64, and the compressors' defining identities."""
import os

import numpy as np
import pytest

import oracle

F32 = np.float32
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    out = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for ln in f:
            if ln.strip() and not ln.startswith("#"):
                parts = ln.split()
                out.setdefault(parts[0], []).append(parts[1:])
    return out


# ------------------------------------------------------------------ Rand-K --

def test_randk_keys_are_the_published_splitmix64_outputs():
    # Seed 0, t = 0: key p = output p >> 40 of the published generator.
    rows = [ln.split() for ln in open(os.path.join(GOLDEN, "splitmix64_seed0.txt"))
            if ln.strip() and not ln.startswith("#")]
    want = np.array([float(int(x, 16) >> 40) for _, x in rows], F32)
    assert np.array_equal(oracle.randk_keys(0, 0, len(want)), want)
    # t advances the counter by m: key p at t equals key t*m + p at t = 0.
    m = 7
    assert np.array_equal(oracle.randk_keys(0, 2, m), oracle.randk_keys(0, 0, 3 * m)[2 * m:])


def test_randk_selects_k_rows_independent_of_the_gradient():
    N, n, m, K = 3, 8, 50, 9
    d = n * m
    rng = np.random.default_rng(0)
    outs = []
    for _ in range(2):
        h, g = np.zeros((N, d), F32), np.zeros((N, d), F32)
        grad = rng.standard_normal((N, d)).astype(F32)
        outs.append(oracle.step_randk(h, g, grad, eta=1.0, seed=11, t=4, n=n, K=K))
    idx = outs[0]["idx"]
    assert np.array_equal(idx, outs[1]["idx"])
    assert len(set(idx.tolist())) == K and np.all(np.diff(idx) > 0)
    keys = oracle.randk_keys(11, 4, m)
    assert set(idx.tolist()) == set(np.argsort(-keys.astype(np.float64), kind="stable")[:K])


def test_randk_payload_and_ef_update_brute_force():
    N, n, m, K, eta = 4, 16, 30, 6, 0.5
    d = n * m - 5  # ragged last row
    rng = np.random.default_rng(1)
    h = rng.standard_normal((N, d)).astype(F32)
    g = rng.standard_normal((N, d)).astype(F32)
    grad = rng.standard_normal((N, d)).astype(F32)
    h0, g0 = h.copy(), g.copy()
    out = oracle.step_randk(h, g, grad, eta=eta, seed=3, t=1, n=n, K=K)
    hn = (np.float32(eta) * grad + (np.float32(1) - np.float32(eta)) * h0).astype(F32)
    assert np.allclose(h, hn, rtol=1e-6, atol=1e-6)
    delta = h - g0
    for q, p in enumerate(out["idx"]):
        lo, hi = p * n, min(p * n + n, d)
        want = delta[:, lo:hi].astype(np.float64).sum(axis=0)
        assert np.allclose(out["agg"][q, : hi - lo], want, rtol=1e-5, atol=1e-6)
        assert np.all(out["agg"][q, hi - lo:] == 0)
        assert np.array_equal(g[:, lo:hi], (g0[:, lo:hi] + delta[:, lo:hi]).astype(F32))
    untouched = np.ones(d, bool)
    for p in out["idx"]:
        untouched[p * n: p * n + n] = False
    assert np.array_equal(g[:, untouched], g0[:, untouched])


def test_randk_uniform_and_contractive_in_expectation():
    # Each row kept with probability K/m; E||C(x) - x||^2 = (1 - K/m)||x||^2
    # (unscaled Rand-K), checked over 2000 draws of the shared seed's stream.
    N, n, m, K, T = 1, 1, 40, 10, 2000
    x = np.linspace(-2, 2, m).astype(F32)
    counts = np.zeros(m)
    err = 0.0
    for t in range(T):
        h = x[None, :].copy()
        g = np.zeros((N, m), F32)
        out = oracle.step_randk(h, g, x[None, :], eta=1.0, seed=99, t=t, n=n, K=K)
        counts[out["idx"]] += 1
        kept = np.zeros(m, bool)
        kept[out["idx"]] = True
        err += float(np.sum(x[~kept].astype(np.float64) ** 2))
    p_hat = counts / T
    assert np.all(np.abs(p_hat - K / m) < 5 * np.sqrt(K / m * (1 - K / m) / T))
    want = (1 - K / m) * float(np.sum(x.astype(np.float64) ** 2))
    assert abs(err / T - want) < 0.03 * want


def test_randk_tensors_select_per_tensor():
    tensors = [(20, 8, 3), (1, 5, 1), (15, 4, 15), (30, 2, 0)]
    d = sum(r * c for r, c, _ in tensors)
    N = 2
    rng = np.random.default_rng(2)
    h, g = np.zeros((N, d), F32), np.zeros((N, d), F32)
    grad = rng.standard_normal((N, d)).astype(F32)
    out = oracle.step_randk(h, g, grad, eta=1.0, seed=5, t=0, tensors=tensors, want_keys=True)
    idx = out["idx"]
    assert len(idx) == 3 + 1 + 15
    assert np.all((idx[:3] >= 0) & (idx[:3] < 20)) and idx[3] == 20
    assert np.array_equal(idx[4:], np.arange(21, 36))
    assert out["agg"].shape == (3 * 8 + 5 + 15 * 4,)


# ------------------------------------------------------------------- Top-K --

def test_topk_prop1_worked_example():
    gd = _golden("prop1_example.txt")
    grad = np.array([[float(v) for v in gd["grad0"][0]], [float(v) for v in gd["grad1"][0]]], F32)
    h, g = np.zeros((2, 2), F32), np.zeros((2, 2), F32)
    out = oracle.step_topk(h, g, grad, eta=1.0, n=1, K=1)
    # merge the gathered payloads: node i's row idx[i][0] carries agg[i][0]
    merged = np.zeros(2)
    for i in range(2):
        merged[out["idx"][i, 0]] += out["agg"][i, 0]
    mean = merged / 2
    assert np.array_equal(mean, np.array([float(v) for v in gd["local_topk_mean"][0]]))
    g_mean = grad.astype(np.float64).mean(axis=0)
    assert np.sum((mean - g_mean) ** 2) == pytest.approx(np.sum(g_mean ** 2))


def test_topk_rows_are_each_nodes_largest_norms_brute_force():
    N, n, m, K = 4, 12, 60, 7
    d = n * m - 3
    rng = np.random.default_rng(3)
    h = rng.standard_normal((N, d)).astype(F32)
    g = rng.standard_normal((N, d)).astype(F32)
    grad = rng.standard_normal((N, d)).astype(F32)
    g0 = g.copy()
    out = oracle.step_topk(h, g, grad, eta=0.3, n=n, K=K, want_norms=True)
    delta = (h - g0).astype(np.float64)
    pad = np.zeros((N, m * n))
    pad[:, :d] = delta
    norms64 = (pad.reshape(N, m, n) ** 2).sum(axis=2)
    assert np.allclose(out["norms"], norms64, rtol=1e-5)
    for i in range(N):
        want = np.sort(np.argsort(-norms64[i], kind="stable")[:K])
        assert np.array_equal(out["idx"][i], want), i
        for q, p in enumerate(out["idx"][i]):
            lo, hi = p * n, min(p * n + n, d)
            row = out["agg"][i].reshape(K, n)[q]
            assert np.array_equal(row[: hi - lo], (h[i, lo:hi] - g0[i, lo:hi]).astype(F32))
            assert np.all(row[hi - lo:] == 0)
    # g moves on each node's own rows only
    for i in range(N):
        own = np.zeros(d, bool)
        for p in out["idx"][i]:
            own[p * n: p * n + n] = True
        assert np.array_equal(g[i, ~own], g0[i, ~own])
        assert np.array_equal(g[i, own], (g0[i, own] + (h[i, own] - g0[i, own])).astype(F32))


def test_topk_norm_chain_order():
    # The squared norm is an fmaf chain in ascending column order from +0.
    # Row [1, 2^-12 x 4]: in that order each 2^-24 is a half ulp of 1 and
    # rounds away (ties to even), giving exactly 1; summing the small squares
    # first (descending order, or pairwise) would give 1 + 2^-22.
    row = np.array([1.0] + [2.0**-12] * 4, F32)
    out = oracle.step_topk(row[None, :].copy(), np.zeros((1, 5), F32), row[None, :], eta=1.0,
                           n=5, K=1, want_norms=True)
    assert out["norms"][0, 0] == np.float32(1.0)
    assert np.float32(np.float32(4 * 2.0**-24) + np.float32(1.0)) == np.float32(1 + 2.0**-22)


def test_topk_tensors_equal_single_view_when_widths_agree():
    N, n = 3, 16
    tensors = [(20, n, 4), (7, n, 7), (13, n, 2)]
    m = 40
    d = m * n
    rng = np.random.default_rng(4)
    grad = rng.standard_normal((N, d)).astype(F32)
    h1, g1 = np.zeros((N, d), F32), np.zeros((N, d), F32)
    h2, g2 = h1.copy(), g1.copy()
    a = oracle.step_topk(h1, g1, grad, eta=0.5, tensors=tensors)
    b = oracle.step_topk(h2, g2, grad, eta=0.5, n=n, buckets=([0, 20, 27, 40], [4, 7, 2]))
    assert np.array_equal(a["idx"], b["idx"])
    assert np.array_equal(a["agg"], b["agg"])
    assert np.array_equal(g1, g2)


def test_topk_single_node_is_the_exact_row_top_k():
    # N = 1: the node's own rows of largest ||Delta_p||^2 are the exact row
    # top-K that ARC-Top-K approximates with its sketch.
    n, m, K = 8, 100, 10
    rng = np.random.default_rng(5)
    x = rng.standard_normal((1, n * m)).astype(F32)
    out = oracle.step_topk(np.zeros_like(x), np.zeros_like(x), x, eta=1.0, n=n, K=K)
    norms = (x.astype(np.float64).reshape(m, n) ** 2).sum(axis=1)
    assert np.array_equal(out["idx"][0], np.sort(np.argsort(-norms)[:K]))


# ---------------------------------------------------- Top-K merge into G --

def test_topk_merge_prop1_worked_example():
    # Prop. 1: the merged local selections cancel; G (the node sum) stays
    # [0, 0] while the sum of the gradients is [0, 0.2]: C(g) = 0, so the
    # error is ||g||^2.
    gd = _golden("prop1_example.txt")
    grad = np.array([[float(v) for v in gd["grad0"][0]], [float(v) for v in gd["grad1"][0]]], F32)
    h, g = np.zeros((2, 2), F32), np.zeros((2, 2), F32)
    out = oracle.step_topk(h, g, grad, eta=1.0, n=1, K=1)
    G = np.zeros(2, F32)
    oracle.merge_topk(G, out["idx"], out["agg"], n=1)
    mean = G.astype(np.float64) / 2
    assert np.array_equal(mean, np.array([float(v) for v in gd["local_topk_mean"][0]]))
    g_mean = grad.astype(np.float64).mean(axis=0)
    assert np.sum((mean - g_mean) ** 2) == pytest.approx(np.sum(g_mean ** 2))


def test_topk_merge_small_integers_brute_force():
    # Small integers are exact in binary32, so the merge must equal the exact
    # scatter-add of every node's kept rows (overlapping and disjoint rows,
    # a ragged last row).
    rng = np.random.default_rng(12)
    for N, n, m, K in ((3, 5, 40, 9), (5, 8, 12, 12), (2, 1, 30, 30), (4, 7, 20, 1)):
        d = n * m - (n // 2)
        idx = np.stack([np.sort(rng.choice(m, K, replace=False)) for _ in range(N)]).astype(
            np.int32)
        agg = rng.integers(-50, 50, size=(N, K * n)).astype(F32)
        for i in range(N):  # payload past d is +0 (as step_topk writes it)
            for q in range(K):
                p = idx[i, q]
                for j in range(n):
                    if p * n + j >= d:
                        agg[i, q * n + j] = 0.0
        G0 = rng.integers(-1000, 1000, size=d).astype(F32)
        G = G0.copy()
        oracle.merge_topk(G, idx, agg, n=n)
        want = G0.astype(np.int64)
        for i in range(N):
            for q in range(K):
                p = idx[i, q]
                for j in range(n):
                    if p * n + j < d:
                        want[p * n + j] += int(agg[i, q * n + j])
        assert np.array_equal(G.astype(np.int64), want), (N, n, m, K)


def test_topk_merge_sums_nodes_in_ascending_order_before_adding():
    # All three nodes keep row 0 with values 2^24, 1, -2^24: ascending sum
    # (2^24 + 1) - 2^24 rounds to 0 (descending would give 1).  Then with
    # G = 2^24 and two nodes adding 1 each: the sum first gives 2^24 + 2,
    # adding one at a time into G would leave 2^24.
    idx = np.zeros((3, 1), np.int32)
    agg = np.array([[2.0 ** 24], [1.0], [-(2.0 ** 24)]], F32)
    G = np.zeros(1, F32)
    oracle.merge_topk(G, idx, agg, n=1)
    assert G[0] == 0.0
    G = np.array([2.0 ** 24], F32)
    oracle.merge_topk(G, np.zeros((2, 1), np.int32), np.ones((2, 1), F32), n=1)
    assert G[0] == 2.0 ** 24 + 2


def test_topk_merge_with_shared_rows_is_the_shared_row_accumulate():
    # Every node keeping the same rows: the merge equals G += (ascending sum
    # of the payloads) at those rows, the shared-row route.
    rng = np.random.default_rng(13)
    N, n, m, K = 4, 6, 25, 8
    d = n * m
    rows = np.sort(rng.choice(m, K, replace=False)).astype(np.int32)
    idx = np.tile(rows, (N, 1))
    agg = rng.standard_normal((N, K * n)).astype(F32)
    G0 = rng.standard_normal(d).astype(F32)
    G = G0.copy()
    oracle.merge_topk(G, idx, agg, n=n)
    summed = agg[0].copy()
    for i in range(1, N):
        summed = (summed + agg[i]).astype(F32)
    G_shared = G0.copy()
    oracle.accumulate(G_shared, rows, summed, n=n)
    assert np.array_equal(G.view(np.uint32), G_shared.view(np.uint32))


def test_topk_merge_keeping_every_row_is_the_dense_step():
    # K = m: every node keeps every row, so the merged G is the dense step's
    # G (the identity compressor), bit for bit.
    rng = np.random.default_rng(14)
    N, n, m = 3, 8, 20
    d = n * m - 3
    h = rng.standard_normal((N, d)).astype(F32)
    g = rng.standard_normal((N, d)).astype(F32)
    grad = rng.standard_normal((N, d)).astype(F32)
    G0 = rng.standard_normal(d).astype(F32)
    h1, g1, G1 = h.copy(), g.copy(), G0.copy()
    out = oracle.step_topk(h1, g1, grad, eta=0.25, n=n, K=m)
    oracle.merge_topk(G1, out["idx"], out["agg"], n=n)
    h2, g2, G2 = h.copy(), g.copy(), G0.copy()
    oracle.dense_step(h2, g2, G2, grad, 0.25)
    for a, b in ((h1, h2), (g1, g2), (G1, G2)):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_topk_merge_tensors_equal_single_view_when_widths_agree():
    rng = np.random.default_rng(15)
    N, w = 3, 16
    tensors = [(10, w, 3), (7, w, 7), (12, w, 2)]
    m = sum(r for r, _, _ in tensors)
    d = m * w
    h = rng.standard_normal((N, d)).astype(F32)
    g = rng.standard_normal((N, d)).astype(F32)
    grad = rng.standard_normal((N, d)).astype(F32)
    G0 = rng.standard_normal(d).astype(F32)
    ht, gt, Gt = h.copy(), g.copy(), G0.copy()
    out_t = oracle.step_topk(ht, gt, grad, eta=0.5, tensors=tensors)
    oracle.merge_topk(Gt, out_t["idx"], out_t["agg"], tensors=tensors)
    begin = np.cumsum([0] + [r for r, _, _ in tensors]).tolist()
    hb, gb, Gb = h.copy(), g.copy(), G0.copy()
    out_b = oracle.step_topk(hb, gb, grad, eta=0.5, n=w,
                             buckets=(begin, [k for _, _, k in tensors]))
    oracle.merge_topk(Gb, out_b["idx"], out_b["agg"], n=w)
    assert np.array_equal(out_t["idx"], out_b["idx"])
    assert np.array_equal(Gt.view(np.uint32), Gb.view(np.uint32))


def test_topk_merge_rejects_rows_out_of_range_or_repeated():
    G = np.zeros(20, F32)
    with pytest.raises(oracle.OracleError):
        oracle.merge_topk(G, np.array([[0, 5]], np.int32), np.zeros((1, 8), F32), n=4)
    with pytest.raises(oracle.OracleError):
        oracle.merge_topk(G, np.array([[1, 1]], np.int32), np.zeros((1, 8), F32), n=4)
