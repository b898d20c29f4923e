"""GPU parity on seeded random layouts: widths, worker counts, projection
dimensions, K, gradient types and per-tensor mixes drawn from a fixed seed,
each small enough for the oracle, every output compared bit for bit (the
rows kept exactly; h, g and the payload within the 1e-5 bound and, with the
shared operation order, bit for bit)."""
import numpy as np
import pytest
import torch

from parity_util import log, run_case

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _single_view_case(rng):
    n = int(rng.choice([1, 3, 4, 8, 12, 32, 64, 96, 100, 128, 256, 384, 512, 768, 1000, 1024,
                        2048, 2304, 4096]))
    rows = int(rng.integers(1, max(2, 400_000 // n)))
    tail = int(rng.integers(0, n)) if rng.random() < 0.5 else 0
    d = max(1, (rows - (1 if tail else 0)) * n + tail)
    m = -(-d // n)
    N = int(rng.choice([1, 2, 3, 4, 5, 8, 16]))
    r = int(rng.choice([1, 2, 3, 4, 4, 4, 8, 17]))
    K = int(rng.choice([0, 1, max(1, m // 100), max(1, m // 10), m, m + 5]))
    grad_dtype = "bf16" if rng.random() < 0.4 else "f32"
    return dict(d=d, N=N, n=n, r=r, K=K, grad_dtype=grad_dtype,
                family=1 if grad_dtype == "bf16" else 0, eta=float(rng.choice([0.05, 0.1, 0.5])))


def _tensor_case(rng):
    tensors = []
    for _ in range(int(rng.integers(1, 9))):
        cols = int(rng.choice([1, 3, 4, 7, 64, 96, 147, 256, 300, 512, 576, 768, 1152, 2048]))
        rows = int(rng.integers(1, max(2, 60_000 // cols)))
        K = int(rng.choice([0, 1, max(1, rows // 20), rows, rows + 3]))
        tensors.append((rows, cols, K))
    d = sum(a * b for a, b, _ in tensors)
    N = int(rng.choice([1, 2, 3, 4, 8]))
    grad_dtype = "bf16" if rng.random() < 0.4 else "f32"
    return dict(d=d, N=N, tensors=tensors, r=int(rng.choice([2, 4, 4, 8])),
                grad_dtype=grad_dtype, family=1 if grad_dtype == "bf16" else 0, eta=0.1)


CASES = []
_rng = np.random.default_rng(20260)
for _k in range(24):
    CASES.append((f"view{_k}", _single_view_case(_rng)))
for _k in range(12):
    CASES.append((f"tensors{_k}", _tensor_case(_rng)))


@pytest.mark.parametrize("name,kw", CASES, ids=[c[0] for c in CASES])
def test_random_layout_parity(name, kw):
    log(f"[random] {name} {kw if 'tensors' not in kw else dict(kw, tensors=len(kw['tensors']))}")
    run_case(label=name, steps=2, seed=7 + len(name), **kw)


# Pointers 16-byte aligned but 0 to 112 bytes past a 128-byte line (gradient
# kept 16-byte aligned for bf16): rows off the lines take the shifted
# column windows of the 8- and 16-row kernels.
OFFLINE_CASES = []
_orng = np.random.default_rng(20262)
for _k in range(24):
    _kw = _single_view_case(_orng) if _k % 3 else _tensor_case(_orng)
    _mis = int(_orng.choice([0, 4, 8, 12, 16, 20, 24, 28]))
    if _kw["grad_dtype"] == "bf16" and _mis % 8:
        _mis += 4
    OFFLINE_CASES.append((f"offline{_k}_{_mis}", dict(_kw, misalign=_mis)))


@pytest.mark.parametrize("name,kw", OFFLINE_CASES, ids=[c[0] for c in OFFLINE_CASES])
def test_random_layout_off_line_pointers(name, kw):
    log(f"[random] {name}")
    run_case(label=name, steps=2, seed=5 + len(name), check_S="tensors" not in kw, **kw)


from test_gpu_model import run_model_case  # noqa: E402

MODEL_CASES = []
_mrng = np.random.default_rng(20261)
for _k in range(12):
    _kw = _single_view_case(_mrng) if _k % 3 else _tensor_case(_mrng)
    _kw = {k: v for k, v in _kw.items() if k != "eta"}
    _kw["compressor"] = ("arc", "randk", "topk")[_k % 3]
    _kw["optimizer"] = ("sgd", "msgd", "adam", "adam")[_k % 4]
    _kw["dense_steps"] = int(_mrng.integers(0, 2))
    MODEL_CASES.append((f"model{_k}_{_kw['compressor']}_{_kw['optimizer']}", _kw))


@pytest.mark.parametrize("name,kw", MODEL_CASES, ids=[c[0] for c in MODEL_CASES])
def test_random_layout_model_step(name, kw):
    log(f"[random] {name}")
    run_model_case(label=name, steps=3, **kw)
