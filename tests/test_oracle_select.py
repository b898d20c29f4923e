"""Pins for the oracle's arg-top-K (Eq. (4)) with the lower-row tie rule,
checked against a brute-force full sort on tiny inputs."""
import numpy as np
import pytest

import oracle

F32 = np.float32


def brute_topk(sigma, K, lo=0, hi=None):
    hi = len(sigma) if hi is None else hi
    order = sorted(range(lo, hi), key=lambda p: (-float(sigma[p]), p))
    return sorted(order[: max(0, min(K, hi - lo))])


@pytest.mark.parametrize("m", [1, 2, 7, 31, 64])
def test_select_matches_full_sort_with_ties(m):
    rng = np.random.default_rng(m)
    for trial in range(20):
        # few distinct values -> many ties; include zeros and subnormals
        pool = np.array([0.0, 1e-45, 1e-40, 0.5, 1.0, 3.0, 3.0000002, 1e30], F32)
        sigma = rng.choice(pool[: 2 + trial % 7], size=m).astype(F32)
        for K in range(0, m + 3):
            got = oracle.select(sigma, K)
            assert got.tolist() == brute_topk(sigma, K), (m, trial, K)


def test_select_all_equal_takes_lowest_rows():
    sigma = np.full(50, 2.5, F32)
    assert oracle.select(sigma, 7).tolist() == list(range(7))
    assert oracle.select(np.zeros(50, F32), 3).tolist() == [0, 1, 2]


def test_select_k_zero_and_k_at_least_m():
    sigma = np.random.default_rng(0).random(40).astype(F32)
    assert oracle.select(sigma, 0).size == 0
    assert oracle.select(sigma, 40).tolist() == list(range(40))
    assert oracle.select(sigma, 1000).tolist() == list(range(40))


def test_select_ascending_output_large():
    rng = np.random.default_rng(5)
    sigma = rng.random(100_000).astype(F32) ** 3
    idx = oracle.select(sigma, 1234)
    assert np.all(np.diff(idx) > 0)
    # every selected key >= every unselected key
    mask = np.zeros(sigma.size, bool)
    mask[idx] = True
    assert sigma[mask].min() >= sigma[~mask].max()


def test_select_buckets_brute_force():
    rng = np.random.default_rng(6)
    m = 60
    begin = [0, 10, 11, 35, 60]
    ks = [3, 5, 0, 40]  # 5 > 1 row and 40 > 25 rows are clamped
    for _ in range(30):
        sigma = rng.choice(np.array([0, 1, 2, 3], F32), size=m).astype(F32)
        got = oracle.select(sigma, buckets=(begin, ks))
        want = []
        for b in range(4):
            want += brute_topk(sigma, ks[b], begin[b], begin[b + 1])
        assert got.tolist() == want


@pytest.mark.parametrize("begin,ks", [
    ([1, 5, 10], [1, 1]),      # does not start at 0
    ([0, 5, 9], [1, 1]),       # does not end at m
    ([0, 5, 5, 10], [1, 1, 1]),  # empty bucket
    ([0, 5, 10], [1, -1]),     # negative K
])
def test_select_rejects_bad_buckets(begin, ks):
    with pytest.raises(oracle.OracleError):
        oracle.select(np.ones(10, F32), buckets=(begin, ks))


def test_select_rejects_negative_k():
    with pytest.raises(oracle.OracleError):
        oracle.select(np.ones(10, F32), -1)
