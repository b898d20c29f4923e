"""Plain CPU oracle of the ARC-Top-K + EF21M compressor step (ctypes wrapper).

TEST INFRASTRUCTURE ONLY.  Only the tests, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  The product path
(``paper_2510_26709_amd`` / libarctopk) never imports it and shares no code
with it.  Every function here marshals numpy arrays into the C oracle
(``arc_oracle.c``); the arithmetic, and the citation of the paper passage each
step follows, live there.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# ARC_ORACLE_LIB selects another build of the same source (the sanitizer
# test loads an instrumented copy this way).
_LIB_PATH = os.environ.get("ARC_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")
_lib = None

_i32, _i64, _u64, _f32 = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_float
_vp = ctypes.c_void_p


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise ImportError(f"{_LIB_PATH} missing: run __graft_entry__.build() or python oracle/build.py")
    lib = ctypes.CDLL(_LIB_PATH)
    sig = {
        "oracle_splitmix64": (_u64, [_u64, _u64]),
        "oracle_projection": (ctypes.c_int, [_u64, _i64, _i64, _i32, _vp]),
        "oracle_momentum": (ctypes.c_int, [_i32, _i64, _f32, _vp, _i32, _vp]),
        "oracle_sketch": (ctypes.c_int, [_i32, _i64, _i64, _i32, _vp, _vp, _vp, _vp]),
        "oracle_worker_sum": (ctypes.c_int, [_i32, _i64, _i32, _vp, _vp]),
        "oracle_importance": (ctypes.c_int, [_i64, _i32, _vp, _vp]),
        "oracle_select": (ctypes.c_int, [_i64, _vp, _i64, _i32, _vp, _vp, _vp, _vp]),
        "oracle_gather_update": (ctypes.c_int, [_i32, _i64, _i64, _i64, _vp, _vp, _vp, _vp]),
        "oracle_step": (ctypes.c_int, [_i32, _i64, _i64, _i32, _f32, _u64, _i64, _i64, _i32,
                                       _vp, _vp, _vp, _i32, _vp, _vp, _vp, _vp, _vp, _vp,
                                       _vp, _vp]),
        "oracle_step_tensors": (ctypes.c_int, [_i32, _i32, _f32, _u64, _i64, _i32, _vp, _vp, _vp,
                                               _vp, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                               _vp]),
        "oracle_dense_step": (ctypes.c_int, [_i32, _i64, _f32, _vp, _i32, _vp, _vp, _vp]),
        "oracle_accumulate_rows": (ctypes.c_int, [_i64, _i64, _i64, _vp, _vp, _vp]),
        "oracle_accumulate_tensors": (ctypes.c_int, [_i32, _vp, _vp, _vp, _vp, _vp, _vp]),
        "oracle_optimizer": (ctypes.c_int, [_i32, _i32, _i64, _i64, _f32, _f32, _f32, _f32, _f32,
                                            _f32, _vp, _vp, _vp, _vp]),
        "oracle_randk_keys": (ctypes.c_int, [_u64, _i64, _i64, _vp]),
        "oracle_step_randk": (ctypes.c_int, [_i32, _i64, _i64, _f32, _u64, _i64, _i64, _i32, _vp,
                                             _vp, _vp, _i32, _vp, _vp, _vp, _vp, _vp, _vp]),
        "oracle_step_randk_tensors": (ctypes.c_int, [_i32, _f32, _u64, _i64, _i32, _vp, _vp, _vp,
                                                     _vp, _i32, _vp, _vp, _vp, _vp, _vp, _vp,
                                                     _vp]),
        "oracle_step_topk": (ctypes.c_int, [_i32, _i64, _i64, _f32, _i64, _i32, _vp, _vp, _vp,
                                            _i32, _vp, _vp, _vp, _vp, _vp, _vp]),
        "oracle_step_topk_tensors": (ctypes.c_int, [_i32, _f32, _i32, _vp, _vp, _vp, _vp, _i32,
                                                    _vp, _vp, _vp, _vp, _vp, _vp, _vp]),
        "oracle_merge_topk_rows": (ctypes.c_int, [_i32, _i64, _i64, _i64, _vp, _vp, _vp]),
        "oracle_merge_topk_tensors": (ctypes.c_int, [_i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp]),
        "oracle_num_threads": (ctypes.c_int, []),
        "oracle_set_num_threads": (None, [ctypes.c_int]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


class OracleError(ValueError):
    pass


def _ptr(a):
    return None if a is None else a.ctypes.data


def _check(rc, what):
    if rc != 0:
        raise OracleError(f"{what}: invalid argument")


def _f32c(a, name):
    if a.dtype != np.float32 or not a.flags.c_contiguous:
        raise TypeError(f"{name} must be a C-contiguous float32 array")
    return a


def _grad_args(grad):
    if grad.dtype == np.float32:
        return grad, 0
    if grad.dtype == np.uint16:  # bf16 bit patterns
        return grad, 1
    raise TypeError("grad must be float32 or uint16 (bf16 bit patterns)")


def num_rows(d: int, n: int) -> int:
    return -(-d // n)


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def set_num_threads(n: int) -> None:
    """Threads of the oracle's parallel loops from now on (results do not
    depend on the count: every row's arithmetic runs in a fixed order)."""
    _load().oracle_set_num_threads(int(n))


def splitmix64(seed: int, x: int) -> int:
    return int(_load().oracle_splitmix64(seed & (2**64 - 1), x & (2**64 - 1)))


def projection(seed: int, t: int, n: int, r: int) -> np.ndarray:
    V = np.empty((n, r), dtype=np.float32)
    _check(_load().oracle_projection(seed & (2**64 - 1), t, n, r, _ptr(V)), "projection")
    return V


def momentum(h: np.ndarray, grad: np.ndarray, eta: float) -> None:
    """In place on h ([N, d] float32)."""
    _f32c(h, "h")
    grad, is_bf16 = _grad_args(np.ascontiguousarray(grad))
    if grad.shape != h.shape:
        raise ValueError("grad and h shapes differ")
    N, d = h.shape
    _check(_load().oracle_momentum(N, d, eta, _ptr(grad), is_bf16, _ptr(h)), "momentum")


def sketch(h: np.ndarray, g: np.ndarray, V: np.ndarray, n: int) -> np.ndarray:
    _f32c(h, "h"), _f32c(g, "g"), _f32c(V, "V")
    N, d = h.shape
    r = V.shape[1]
    if V.shape[0] != n:
        raise ValueError("V must be [n, r]")
    S = np.empty((N, num_rows(d, n), r), dtype=np.float32)
    _check(_load().oracle_sketch(N, d, n, r, _ptr(h), _ptr(g), _ptr(V), _ptr(S)), "sketch")
    return S


def worker_sum(S: np.ndarray) -> np.ndarray:
    _f32c(S, "S")
    N, m, r = S.shape
    P = np.empty((m, r), dtype=np.float32)
    _check(_load().oracle_worker_sum(N, m, r, _ptr(S), _ptr(P)), "worker_sum")
    return P


def importance(P: np.ndarray) -> np.ndarray:
    _f32c(P, "P")
    m, r = P.shape
    sigma = np.empty(m, dtype=np.float32)
    _check(_load().oracle_importance(m, r, _ptr(P), _ptr(sigma)), "importance")
    return sigma


def _bucket_arrays(buckets):
    if buckets is None:
        return 0, None, None
    begin = np.ascontiguousarray(np.asarray(buckets[0], dtype=np.int64))
    kb = np.ascontiguousarray(np.asarray(buckets[1], dtype=np.int64))
    if begin.shape[0] != kb.shape[0] + 1:
        raise ValueError("bucket_row_begin must have num_buckets + 1 entries")
    return kb.shape[0], begin, kb


def select(sigma: np.ndarray, K: int = 0, buckets=None) -> np.ndarray:
    """buckets = (row_begin[nb+1], K[nb]) or None for one global bucket."""
    _f32c(sigma, "sigma")
    m = sigma.shape[0]
    nb, begin, kb = _bucket_arrays(buckets)
    cap = m
    idx = np.empty(cap, dtype=np.int32)
    total = ctypes.c_int64(0)
    _check(_load().oracle_select(m, _ptr(sigma), K, nb, _ptr(begin), _ptr(kb), _ptr(idx),
                                 ctypes.addressof(total)), "select")
    return idx[: total.value].copy()


def gather_update(h: np.ndarray, g: np.ndarray, idx: np.ndarray, n: int) -> np.ndarray:
    """Returns agg [K_total, n]; updates g in place."""
    _f32c(h, "h"), _f32c(g, "g")
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    N, d = h.shape
    agg = np.empty((idx.shape[0], n), dtype=np.float32)
    _check(_load().oracle_gather_update(N, d, n, idx.shape[0], _ptr(idx), _ptr(h), _ptr(g),
                                        _ptr(agg)), "gather_update")
    return agg


def step(h: np.ndarray, g: np.ndarray, grad: np.ndarray, *, n: int, r: int, eta: float,
         seed: int, t: int, K: int = 0, buckets=None, V: np.ndarray | None = None,
         want_sigma: bool = False, want_S: bool = False) -> dict:
    """One compressor step; h and g are updated in place.

    Returns {"idx": int32[K_total], "agg": float32[K_total, n]} plus "sigma" /
    "S" when asked for.
    """
    _f32c(h, "h"), _f32c(g, "g")
    grad, is_bf16 = _grad_args(np.ascontiguousarray(grad))
    N, d = h.shape
    if g.shape != h.shape or grad.shape != h.shape:
        raise ValueError("h, g and grad must all be [N, d]")
    m = num_rows(d, n)
    nb, begin, kb = _bucket_arrays(buckets)
    idx = np.empty(m, dtype=np.int32)
    # Upper bound on the number of selected rows keeps the payload buffer small.
    if nb == 0:
        kmax = min(m, max(K, 0))
    else:
        kmax = int(sum(min(max(int(k), 0), int(b1 - b0))
                       for k, b0, b1 in zip(kb, begin[:-1], begin[1:])))
    agg = np.empty((max(kmax, 1), n), dtype=np.float32)
    sigma = np.empty(m, dtype=np.float32) if want_sigma else None
    S = np.empty((N, m, r), dtype=np.float32) if want_S else None
    if V is not None:
        V = np.ascontiguousarray(V, dtype=np.float32)
        if V.shape != (n, r):
            raise ValueError("V must be [n, r]")
    total = ctypes.c_int64(0)
    _check(_load().oracle_step(N, d, n, r, eta, seed & (2**64 - 1), t, K, nb, _ptr(begin),
                               _ptr(kb), _ptr(grad), is_bf16, _ptr(h), _ptr(g), _ptr(idx),
                               _ptr(agg), ctypes.addressof(total), _ptr(V), _ptr(sigma),
                               _ptr(S)), "step")
    k = total.value
    out = {"idx": idx[:k].copy(), "agg": agg[:k].copy()}
    if want_sigma:
        out["sigma"] = sigma
    if want_S:
        out["S"] = S
    return out


def step_tensors(h: np.ndarray, g: np.ndarray, grad: np.ndarray, tensors, *, r: int, eta: float,
                 seed: int, t: int, want_sigma: bool = False, want_S: bool = False) -> dict:
    """Per-tensor step; tensors = [(rows, cols, K), ...] laid out consecutively.

    Returns {"idx": int32[K_total] (global rows), "agg": float32[agg_len] (packed
    rows of each tensor's width)} plus "sigma" / "S" when asked for.
    """
    _f32c(h, "h"), _f32c(g, "g")
    grad, is_bf16 = _grad_args(np.ascontiguousarray(grad))
    N, d = h.shape
    tens = np.asarray(tensors, dtype=np.int64).reshape(-1, 3)
    rows = np.ascontiguousarray(tens[:, 0])
    cols = np.ascontiguousarray(tens[:, 1])
    ks = np.ascontiguousarray(tens[:, 2])
    if int((rows * cols).sum()) != d or g.shape != h.shape or grad.shape != h.shape:
        raise ValueError("tensors must cover d exactly; h, g, grad must be [N, d]")
    m = int(rows.sum())
    kept = np.minimum(np.maximum(ks, 0), rows)
    idx = np.empty(max(int(kept.sum()), 1), dtype=np.int32)
    agg = np.empty(max(int((kept * cols).sum()), 1), dtype=np.float32)
    sigma = np.empty(m, dtype=np.float32) if want_sigma else None
    S = np.empty((N, m, r), dtype=np.float32) if want_S else None
    total = ctypes.c_int64(0)
    alen = ctypes.c_int64(0)
    _check(_load().oracle_step_tensors(N, r, eta, seed & (2**64 - 1), t, len(rows), _ptr(rows),
                                       _ptr(cols), _ptr(ks), _ptr(grad), is_bf16, _ptr(h),
                                       _ptr(g), _ptr(idx), _ptr(agg), ctypes.addressof(total),
                                       ctypes.addressof(alen), _ptr(sigma), _ptr(S)),
           "step_tensors")
    out = {"idx": idx[: total.value].copy(), "agg": agg[: alen.value].copy()}
    if want_sigma:
        out["sigma"] = sigma
    if want_S:
        out["S"] = S
    return out


# ---- model step around the compressor (Eq. (11c), optimisers, warm-up) ----

OPTIMIZERS = {"sgd": 0, "msgd": 1, "adam": 2}


def dense_step(h: np.ndarray, g: np.ndarray, G: np.ndarray, grad: np.ndarray, eta: float) -> None:
    """Identity-compressor step in place: (11a), (11b) with C = I, G += payload."""
    _f32c(h, "h"), _f32c(g, "g"), _f32c(G, "G")
    grad, is_bf16 = _grad_args(np.ascontiguousarray(grad))
    N, d = h.shape
    if g.shape != h.shape or grad.shape != h.shape or G.shape != (d,):
        raise ValueError("h, g, grad must be [N, d]; G must be [d]")
    _check(_load().oracle_dense_step(N, d, eta, _ptr(grad), is_bf16, _ptr(h), _ptr(g), _ptr(G)),
           "dense_step")


def accumulate(G: np.ndarray, idx: np.ndarray, agg: np.ndarray, *, n: int = 0,
               tensors=None) -> None:
    """G += agg at the selected rows (single view of width n, or tensors)."""
    _f32c(G, "G")
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    agg = np.ascontiguousarray(agg, dtype=np.float32).reshape(-1)
    if tensors is None:
        _check(_load().oracle_accumulate_rows(G.shape[0], n, idx.shape[0], _ptr(idx), _ptr(agg),
                                              _ptr(G)), "accumulate")
    else:
        tens = np.asarray(tensors, dtype=np.int64).reshape(-1, 3)
        rows, cols, ks = (np.ascontiguousarray(tens[:, c]) for c in range(3))
        _check(_load().oracle_accumulate_tensors(len(rows), _ptr(rows), _ptr(cols), _ptr(ks),
                                                 _ptr(idx), _ptr(agg), _ptr(G)), "accumulate")


def merge_topk(G: np.ndarray, idx: np.ndarray, agg: np.ndarray, *, n: int = 0,
               tensors=None) -> None:
    """Top-K's merge into G (in place): idx [N, K_node] and agg [N, L] as
    step_topk returns them; for every coordinate, the values of the nodes that
    kept its row, summed in ascending node order, are added to G."""
    _f32c(G, "G")
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    agg = np.ascontiguousarray(agg, dtype=np.float32)
    if idx.ndim != 2 or agg.ndim != 2 or idx.shape[0] != agg.shape[0]:
        raise ValueError("idx must be [N, K_node] and agg [N, L]")
    N = idx.shape[0]
    if tensors is None:
        if agg.shape[1] != idx.shape[1] * n:
            raise ValueError("agg must hold K_node rows of n values per node")
        _check(_load().oracle_merge_topk_rows(N, G.shape[0], n, idx.shape[1], _ptr(idx),
                                              _ptr(agg), _ptr(G)), "merge_topk")
    else:
        rows, cols, ks = _tensor_arrays(tensors)
        _check(_load().oracle_merge_topk_tensors(N, len(rows), _ptr(rows), _ptr(cols), _ptr(ks),
                                                 _ptr(idx), _ptr(agg), _ptr(G)), "merge_topk")


def optimizer_step(name: str, G: np.ndarray, x: np.ndarray, m=None, v=None, *, N: int, T: int,
                   lr: float, momentum: float = 0.0, beta1: float = 0.9, beta2: float = 0.999,
                   eps: float = 1e-8, weight_decay: float = 0.0) -> None:
    """x (and the optimiser state m, v) updated in place from G."""
    _f32c(G, "G"), _f32c(x, "x")
    for a, nm in ((m, "m"), (v, "v")):
        if a is not None:
            _f32c(a, nm)
    _check(_load().oracle_optimizer(OPTIMIZERS[name], N, x.shape[0], T, lr, momentum, beta1,
                                    beta2, eps, weight_decay, _ptr(G), _ptr(x), _ptr(m),
                                    _ptr(v)), "optimizer")


# ---- comparison compressors of Table I (Rand-K, Top-K) ----

def randk_keys(seed: int, t: int, m: int) -> np.ndarray:
    keys = np.empty(m, dtype=np.float32)
    _check(_load().oracle_randk_keys(seed & (2**64 - 1), t, m, _ptr(keys)), "randk_keys")
    return keys


def _tensor_arrays(tensors):
    tens = np.asarray(tensors, dtype=np.int64).reshape(-1, 3)
    return tuple(np.ascontiguousarray(tens[:, c]) for c in range(3))


def _kept_rows(m, K, buckets, tensors):
    if tensors is not None:
        return int(sum(min(max(int(k), 0), int(r)) for r, _, k in tensors))
    if buckets is None:
        return min(m, max(K, 0))
    begin, kb = buckets
    return int(sum(min(max(int(k), 0), int(b1 - b0)) for k, b0, b1 in
                   zip(kb, begin[:-1], begin[1:])))


def step_randk(h: np.ndarray, g: np.ndarray, grad: np.ndarray, *, eta: float, seed: int, t: int,
               n: int = 0, K: int = 0, buckets=None, tensors=None,
               want_keys: bool = False) -> dict:
    """Rand-K inside the EF21M step (in place on h, g): {"idx", "agg"} as for
    step / step_tensors, plus "keys" when asked for."""
    _f32c(h, "h"), _f32c(g, "g")
    grad, is_bf16 = _grad_args(np.ascontiguousarray(grad))
    N, d = h.shape
    if g.shape != h.shape or grad.shape != h.shape:
        raise ValueError("h, g and grad must all be [N, d]")
    total, alen = ctypes.c_int64(0), ctypes.c_int64(0)
    if tensors is None:
        m = num_rows(d, n)
        kmax = _kept_rows(m, K, buckets, None)
        idx = np.empty(max(m, 1), dtype=np.int32)
        agg = np.empty((max(kmax, 1), n), dtype=np.float32)
        keys = np.empty(m, dtype=np.float32)
        nb, begin, kb = _bucket_arrays(buckets)
        _check(_load().oracle_step_randk(N, d, n, eta, seed & (2**64 - 1), t, K, nb, _ptr(begin),
                                         _ptr(kb), _ptr(grad), is_bf16, _ptr(h), _ptr(g),
                                         _ptr(idx), _ptr(agg), ctypes.addressof(total),
                                         _ptr(keys)), "step_randk")
        out = {"idx": idx[: total.value].copy(), "agg": agg[: total.value].copy()}
    else:
        rows, cols, ks = _tensor_arrays(tensors)
        m = int(rows.sum())
        kmax = _kept_rows(m, 0, None, tensors)
        idx = np.empty(max(m, 1), dtype=np.int32)
        agg = np.empty(max(int(sum(min(max(int(k), 0), int(r)) * int(c)
                                   for r, c, k in tensors)), 1), dtype=np.float32)
        keys = np.empty(m, dtype=np.float32)
        _check(_load().oracle_step_randk_tensors(N, eta, seed & (2**64 - 1), t, len(rows),
                                                 _ptr(rows), _ptr(cols), _ptr(ks), _ptr(grad),
                                                 is_bf16, _ptr(h), _ptr(g), _ptr(idx), _ptr(agg),
                                                 ctypes.addressof(total), ctypes.addressof(alen),
                                                 _ptr(keys)), "step_randk_tensors")
        out = {"idx": idx[: total.value].copy(), "agg": agg[: alen.value].copy()}
    if want_keys:
        out["keys"] = keys
    return out


def step_topk(h: np.ndarray, g: np.ndarray, grad: np.ndarray, *, eta: float, n: int = 0,
              K: int = 0, buckets=None, tensors=None, want_norms: bool = False) -> dict:
    """Local Top-K inside the EF21M step (in place on h, g): {"idx": int32
    [N, K_total] (each node's rows), "agg": float32 [N, L] (each node's own
    rows of Delta, nothing summed)}, plus "norms" [N, m] when asked for."""
    _f32c(h, "h"), _f32c(g, "g")
    grad, is_bf16 = _grad_args(np.ascontiguousarray(grad))
    N, d = h.shape
    if g.shape != h.shape or grad.shape != h.shape:
        raise ValueError("h, g and grad must all be [N, d]")
    total, alen = ctypes.c_int64(0), ctypes.c_int64(0)
    if tensors is None:
        m = num_rows(d, n)
        kmax = _kept_rows(m, K, buckets, None)
        idx = np.empty(max(N * m, 1), dtype=np.int32)
        agg = np.empty(max(N * kmax * n, 1), dtype=np.float32)
        norms = np.empty((N, m), dtype=np.float32)
        nb, begin, kb = _bucket_arrays(buckets)
        _check(_load().oracle_step_topk(N, d, n, eta, K, nb, _ptr(begin), _ptr(kb), _ptr(grad),
                                        is_bf16, _ptr(h), _ptr(g), _ptr(idx), _ptr(agg),
                                        ctypes.addressof(total), _ptr(norms)), "step_topk")
        L = total.value * n
    else:
        rows, cols, ks = _tensor_arrays(tensors)
        m = int(rows.sum())
        Lmax = int(sum(min(max(int(k), 0), int(r)) * int(c) for r, c, k in tensors))
        idx = np.empty(max(N * m, 1), dtype=np.int32)
        agg = np.empty(max(N * Lmax, 1), dtype=np.float32)
        norms = np.empty((N, m), dtype=np.float32)
        _check(_load().oracle_step_topk_tensors(N, eta, len(rows), _ptr(rows), _ptr(cols),
                                                _ptr(ks), _ptr(grad), is_bf16, _ptr(h), _ptr(g),
                                                _ptr(idx), _ptr(agg), ctypes.addressof(total),
                                                ctypes.addressof(alen), _ptr(norms)),
               "step_topk_tensors")
        L = alen.value
    kt = total.value
    out = {"idx": idx[: N * kt].reshape(N, kt).copy(), "agg": agg[: N * L].reshape(N, L).copy()}
    if want_norms:
        out["norms"] = norms
    return out
