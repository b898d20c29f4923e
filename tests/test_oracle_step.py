"""Whole-step pins for the oracle: the paper's worked example (Prop. 1), a
hand-worked EF21M run, the identity case K = m, the shared index set, the
contraction of Prop. 2, the unbiasedness identity Eq. (6), resume and
thread-count invariance."""
import math
import os
import subprocess
import sys

import numpy as np
import pytest

import oracle

F32 = np.float32
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _golden(name):
    out = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for ln in f:
            if ln.strip() and not ln.startswith("#"):
                parts = ln.split()
                out.setdefault(parts[0], []).append(parts[1:])
    return out


# ------------------------------------------------------------ Prop. 1 ------
def test_prop1_worked_example():
    gd = _golden("prop1_example.txt")
    N, d, K = int(gd["N"][0][0]), int(gd["d"][0][0]), int(gd["K"][0][0])
    grad = np.array([[float(x) for x in gd["grad0"][0]], [float(x) for x in gd["grad1"][0]]], F32)
    mean = np.array([float(x) for x in gd["mean"][0]])
    local_topk = np.array([float(x) for x in gd["local_topk_mean"][0]])
    row = int(gd["arc_selected_row"][0][0])
    # the paper's foil: local Top-K then averaging loses everything
    assert np.sum((local_topk - mean) ** 2) == pytest.approx(np.sum(mean ** 2))
    for seed in range(50):  # any shared V selects the non-cancelling row
        h = np.zeros((N, d), F32)
        g = np.zeros((N, d), F32)
        out = oracle.step(h, g, grad, n=1, r=4, eta=1.0, seed=seed, t=0, K=K)
        assert out["idx"].tolist() == [row]
        C = np.zeros(d)
        C[out["idx"]] = out["agg"][:, 0] / N
        assert np.allclose(C, mean, rtol=0, atol=1e-7)
        assert np.sum((C - mean) ** 2) < 1e-12


# ------------------------------------------------- hand-worked EF21M -------
def test_two_step_hand_worked_run():
    rows = _golden("ef21m_two_steps.txt")["step"]
    by = {}
    for r in rows:
        by[(int(r[0]), r[1])] = np.array([float(x) for x in r[2:]], F32)
    N, d, n = 2, 4, 2
    h = np.zeros((N, d), F32)
    g = np.zeros((N, d), F32)
    V = np.ones((2, 1), F32)
    for t in (1, 2):
        out = oracle.step(h, g, by[(t, "grad")].reshape(N, d), n=n, r=1, eta=0.5, seed=0,
                          t=t, K=1, V=V, want_sigma=True)
        assert h.ravel().tolist() == by[(t, "h")].tolist()
        assert out["sigma"].tolist() == by[(t, "sigma")].tolist()
        assert out["idx"].tolist() == by[(t, "idx")].astype(int).tolist()
        assert out["agg"].ravel().tolist() == by[(t, "agg")].tolist()
        assert g.ravel().tolist() == by[(t, "g")].tolist()


def _random_state(rng, N, d, scale_rows=None, n=None):
    grad = rng.standard_normal((N, d)).astype(F32)
    if scale_rows is not None:
        grad = (grad.reshape(N, -1, n) * scale_rows[None, :, None]).reshape(N, d).astype(F32)
    return grad


# ----------------------------------------------------------- identity ------
def test_k_equal_m_is_identity_compressor():
    rng = np.random.default_rng(7)
    N, d, n = 4, 4096, 64
    m = d // n
    h = rng.standard_normal((N, d)).astype(F32)
    g = rng.standard_normal((N, d)).astype(F32)
    grad = rng.standard_normal((N, d)).astype(F32)
    h_before, g_before = h.copy(), g.copy()
    out = oracle.step(h, g, grad, n=n, r=4, eta=0.1, seed=3, t=1, K=m)
    assert out["idx"].tolist() == list(range(m))
    delta = (h - g_before)  # new h minus old g, binary32
    # agg is the ascending-order worker sum of Delta, everywhere
    acc = delta[0].copy()
    for i in range(1, N):
        acc = (acc + delta[i]).astype(F32)
    assert np.array_equal(out["agg"].ravel(), acc)
    # g moved by exactly Delta on every row, so g_t = fl(g + fl(h - g)) is h up
    # to two roundings: |g_t - h| <= 2u (|h| + |g_{t-1}|)
    assert np.array_equal(g, (g_before + delta).astype(F32))
    bound = 2 * 2.0 ** -24 * (np.abs(h).astype(np.float64) + np.abs(g_before))
    assert np.all(np.abs(g.astype(np.float64) - h) <= bound)
    # ||C(x) - x|| = 0 with x the worker mean of Delta
    x = delta.astype(np.float64).mean(axis=0)
    Cx = out["agg"].astype(np.float64).ravel() / N
    assert np.max(np.abs(Cx - x)) <= 4 * 2 ** -24 * np.max(np.abs(delta))
    assert not np.array_equal(h, h_before)


# ------------------------------------------------- shared index set --------
def test_every_worker_moves_only_on_the_shared_rows():
    rng = np.random.default_rng(8)
    N, d, n, K = 4, 1000, 8, 13  # ragged: m = 125 (exact); use d = 1003 below too
    for d in (1000, 1003):
        m = -(-d // n)
        h = rng.standard_normal((N, d)).astype(F32)
        g = rng.standard_normal((N, d)).astype(F32)
        grad = rng.standard_normal((N, d)).astype(F32)
        g_before = g.copy()
        out = oracle.step(h, g, grad, n=n, r=4, eta=0.2, seed=9, t=4, K=K)
        idx = out["idx"]
        assert len(idx) == K and np.all(np.diff(idx) > 0) and idx.max() < m
        sel = np.zeros(m, bool)
        sel[idx] = True
        pad = np.zeros((N, m * n), F32)
        pad[:, :d] = g - g_before
        moved = np.any(pad.reshape(N, m, n) != 0, axis=2)  # [N, m]
        for i in range(N):
            assert not np.any(moved[i] & ~sel), "a worker changed an unselected row"
        # on the selected rows the change is the residual Delta^(i)
        delta = (h - g_before)
        padd = np.zeros((N, m * n), F32)
        padd[:, :d] = delta
        chg = pad.reshape(N, m, n)[:, idx]
        np.testing.assert_allclose(chg, padd.reshape(N, m, n)[:, idx], rtol=2 ** -22, atol=1e-6)


# --------------------------------------------------- Prop. 2 contraction ---
def _contraction_ratio(out, delta, N, n, d):
    x = delta.astype(np.float64).mean(axis=0)
    m = -(-d // n)
    C = np.zeros(m * n)
    C.reshape(m, n)[out["idx"]] = out["agg"].astype(np.float64) / N
    err = np.sum((C[:d] - x) ** 2)
    return err / np.sum(x ** 2), x, C[:d]


def test_contraction_in_expectation_over_the_projection():
    # Prop. 2: E_V ||C(x) - x||^2 <= (1 - K/m) ||x||^2.  Rows of very different
    # size make a wrong selection (or an inverted one) break the bound.
    rng = np.random.default_rng(10)
    N, n, m, K = 4, 16, 32, 4
    d = m * n
    row_scale = np.geomspace(0.05, 3.0, m)[rng.permutation(m)]
    grad = _random_state(rng, N, d, row_scale, n)
    ratios = []
    for seed in range(1000):
        h = np.zeros((N, d), F32)
        g = np.zeros((N, d), F32)
        out = oracle.step(h, g, grad, n=n, r=4, eta=1.0, seed=seed, t=0, K=K)
        ratio, _, _ = _contraction_ratio(out, h, N, n, d)
        ratios.append(ratio)
    ratios = np.array(ratios)
    se = ratios.std(ddof=1) / math.sqrt(len(ratios))
    assert ratios.mean() <= 1 - K / m + 3 * se
    # the sketch really selects large rows: far better than the bound
    assert ratios.mean() < 0.5 * (1 - K / m)


def test_contraction_error_identity_per_draw():
    # ||C(x) - x||^2 = sum over unselected rows of ||x_p||^2, for every draw
    rng = np.random.default_rng(11)
    N, n, d, K = 3, 10, 997, 17
    for seed in range(20):
        grad = rng.standard_normal((N, d)).astype(F32)
        h = np.zeros((N, d), F32)
        g = np.zeros((N, d), F32)
        out = oracle.step(h, g, grad, n=n, r=4, eta=1.0, seed=seed, t=0, K=K)
        _, x, C = _contraction_ratio(out, h, N, n, d)
        m = -(-d // n)
        xp = np.zeros(m * n)
        xp[:d] = x
        keep = np.zeros(m, bool)
        keep[out["idx"]] = True
        rest = np.sum(xp.reshape(m, n)[~keep] ** 2)
        assert np.sum((C - x) ** 2) == pytest.approx(rest, rel=1e-5, abs=1e-9)


def test_exact_sketch_mode_is_global_topk_per_draw():
    # n = 1, r = 1, V = [1]: Sigma_p = (sum_i Delta_i[p])^2, so the selection is
    # the textbook Top-K of |sum_i Delta_i| and contracts on every draw.
    rng = np.random.default_rng(12)
    N, d, K = 4, 300, 30
    for trial in range(10):
        grad = rng.integers(-20, 21, size=(N, d)).astype(F32)
        h = np.zeros((N, d), F32)
        g = np.zeros((N, d), F32)
        out = oracle.step(h, g, grad, n=1, r=1, eta=1.0, seed=0, t=0, K=K, V=np.ones((1, 1), F32))
        tot = np.abs(grad.astype(np.int64).sum(axis=0))
        want = sorted(sorted(range(d), key=lambda p: (-tot[p], p))[:K])
        assert out["idx"].tolist() == want
        ratio, _, _ = _contraction_ratio(out, h, N, 1, d)
        assert ratio <= 1 - K / d + 1e-12


# ------------------------------------------------------ Eq. (6) unbiased ---
def test_importance_is_unbiased_for_row_norm():
    # With the 1/sqrt(r) and 1/N factors left out, Sigma_p = ||sum_i u_p^(i) V||^2
    # so E_V[Sigma_p] = r N^2 ||u_p||^2 with u_p the worker-mean row (Eq. (6)).
    rng = np.random.default_rng(13)
    N, n, m, r = 3, 24, 6, 4
    d = n * m
    grad = rng.standard_normal((N, d)).astype(F32)
    u = grad.astype(np.float64).mean(axis=0).reshape(m, n)
    target = r * N * N * np.sum(u ** 2, axis=1)
    samples = []
    for t in range(4000):
        h = np.zeros((N, d), F32)
        g = np.zeros((N, d), F32)
        out = oracle.step(h, g, grad, n=n, r=r, eta=1.0, seed=99, t=t, K=0, want_sigma=True)
        samples.append(out["sigma"].astype(np.float64))
    samples = np.array(samples)
    mean = samples.mean(axis=0)
    se = samples.std(axis=0, ddof=1) / math.sqrt(samples.shape[0])
    assert np.all(np.abs(mean - target) <= 4 * se)
    # Var of a chi-square with r dof scaled: Var = 2 r (N^2 ||u||^2)^2
    var_target = 2 * r * (N * N * np.sum(u ** 2, axis=1)) ** 2
    np.testing.assert_allclose(samples.var(axis=0), var_target, rtol=0.15)


# --------------------------------------------------------- ties, zeros -----
def test_zero_residual_selects_first_rows():
    N, d, n = 2, 64, 4
    h = np.zeros((N, d), F32)
    g = np.zeros((N, d), F32)
    out = oracle.step(h, g, np.zeros((N, d), F32), n=n, r=4, eta=0.5, seed=1, t=0, K=5,
                      want_sigma=True)
    assert out["idx"].tolist() == [0, 1, 2, 3, 4]
    assert not np.any(out["sigma"])
    assert not np.any(out["agg"])


def test_bucketed_step_selects_per_bucket():
    rng = np.random.default_rng(14)
    N, n, d = 2, 8, 8 * 40
    begin, ks = [0, 10, 30, 40], [2, 3, 10]
    grad = rng.standard_normal((N, d)).astype(F32)
    h = np.zeros((N, d), F32)
    g = np.zeros((N, d), F32)
    out = oracle.step(h, g, grad, n=n, r=4, eta=1.0, seed=5, t=2, buckets=(begin, ks),
                      want_sigma=True)
    idx = out["idx"].tolist()
    assert len(idx) == 15
    s = out["sigma"]
    assert idx[:2] == sorted(sorted(range(0, 10), key=lambda p: (-s[p], p))[:2])
    assert idx[2:5] == sorted(sorted(range(10, 30), key=lambda p: (-s[p], p))[:3])
    assert idx[5:] == list(range(30, 40))


# -------------------------------------------------- resume, determinism ----
def _run(steps, h, g, N, d, seed0=21):
    outs = []
    for t in steps:
        grad = np.random.default_rng(seed0 + t).standard_normal((N, d)).astype(F32)
        outs.append(oracle.step(h, g, grad, n=16, r=4, eta=0.1, seed=4, t=t, K=9))
    return outs


def test_resume_is_bit_identical():
    N, d = 3, 16 * 50 + 5
    h1, g1 = np.zeros((N, d), F32), np.zeros((N, d), F32)
    full = _run(range(10), h1, g1, N, d)
    h2, g2 = np.zeros((N, d), F32), np.zeros((N, d), F32)
    first = _run(range(5), h2, g2, N, d)
    saved_h, saved_g = h2.copy(), g2.copy()
    h3, g3 = saved_h.copy(), saved_g.copy()
    second = _run(range(5, 10), h3, g3, N, d)
    for a, b in zip(full, first + second):
        assert a["idx"].tobytes() == b["idx"].tobytes()
        assert a["agg"].tobytes() == b["agg"].tobytes()
    assert h1.tobytes() == h3.tobytes() and g1.tobytes() == g3.tobytes()


_THREAD_SCRIPT = r"""
import sys, hashlib, numpy as np
sys.path.insert(0, sys.argv[1])
import oracle
rng = np.random.default_rng(3)
N, d = 4, 64 * 997
h = np.zeros((N, d), np.float32); g = np.zeros((N, d), np.float32)
dig = hashlib.sha256()
for t in range(3):
    grad = rng.standard_normal((N, d)).astype(np.float32)
    out = oracle.step(h, g, grad, n=64, r=4, eta=0.1, seed=8, t=t, K=40, want_sigma=True)
    for k in ("idx", "agg", "sigma"):
        dig.update(out[k].tobytes())
dig.update(h.tobytes()); dig.update(g.tobytes())
print(oracle.num_threads(), dig.hexdigest())
"""


def test_thread_count_invariance():
    res = []
    for threads in ("1", "5"):
        env = dict(os.environ, OMP_NUM_THREADS=threads)
        out = subprocess.run([sys.executable, "-c", _THREAD_SCRIPT, ROOT], env=env,
                             capture_output=True, text=True, check=True).stdout.split()
        assert out[0] == threads
        res.append(out[1])
    assert res[0] == res[1]


def test_set_num_threads_changes_only_the_thread_count():
    before = oracle.num_threads()
    rng = np.random.default_rng(5)
    N, d = 2, 32 * 301
    grad = rng.standard_normal((N, d)).astype(F32)
    outs = []
    try:
        for threads in (1, max(2, before)):
            oracle.set_num_threads(threads)
            assert oracle.num_threads() == threads
            h, g = np.zeros((N, d), F32), np.zeros((N, d), F32)
            out = oracle.step(h, g, grad, n=32, r=4, eta=0.3, seed=2, t=1, K=7)
            outs.append((out["idx"].tobytes(), out["agg"].tobytes(), h.tobytes(), g.tobytes()))
    finally:
        oracle.set_num_threads(before)
    assert oracle.num_threads() == before
    assert outs[0] == outs[1]


def test_step_rejects_bad_config_before_touching_state():
    h = np.ones((2, 8), F32)
    g = np.zeros((2, 8), F32)
    with pytest.raises(oracle.OracleError):
        oracle.step(h, g, np.ones((2, 8), F32), n=2, r=4, eta=0.5, seed=0, t=0,
                    buckets=([0, 3, 5], [1, 1]))  # buckets end at 5 != m = 4
    assert np.all(h == 1)
