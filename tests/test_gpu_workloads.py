"""Full-size parity: the five benchmark workloads at their real sizes, and the
per-tensor variants of three of them, every step, in the launch configuration
bench.py times, against the CPU oracle run on the whole workload.

Per step: selected rows and the importance bit-exact; agg bit-exact (and
within 1e-5 relative max-norm); h and g compared on the selected rows plus a
seeded sample of other rows.  After the last step h and g are compared in
full.  Gradients are made on the device by the synthetic generator (whose
bits equal the host generator's, see test_gpu_parity) and copied to the host
for the oracle.
"""
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2510_26709_amd as arc
import synth
from parity_util import compare_float, log, timed

pytestmark = pytest.mark.gpu
F32 = np.float32


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _host_copy(t: torch.Tensor) -> np.ndarray:
    a = t.cpu().numpy()
    return a.view(np.uint16) if a.dtype == np.int16 else a


def _row_spans(w):
    """p -> [lo, hi) coordinate range of row p of the workload's view(s)."""
    if not w.per_tensor:
        return lambda p: (int(p) * w.n, min(int(p) * w.n + w.n, w.d))
    rows = np.array([r for r, _ in w.views], np.int64)
    cols = np.array([c for _, c in w.views], np.int64)
    row0 = np.concatenate([[0], np.cumsum(rows)])
    off = np.concatenate([[0], np.cumsum(rows * cols)])

    def span(p):
        b = int(np.searchsorted(row0, int(p), side="right")) - 1
        lo = int(off[b] + (int(p) - row0[b]) * cols[b])
        return lo, lo + int(cols[b])
    return span


def _compare_rows(label, dev_state, host_state, rows, span):
    """Compare the given rows of an [N, d] state (device) with the oracle's."""
    for p in rows:
        lo, hi = span(p)
        got = dev_state[:, lo:hi].cpu().numpy()
        compare_float(f"{label} row {p}", got, host_state[:, lo:hi])


def _compare_full(label, dev_state, host_state, chunk=1 << 27):
    N, d = host_state.shape
    for i in range(N):
        for lo in range(0, d, chunk):
            hi = min(d, lo + chunk)
            compare_float(f"{label} worker {i} [{lo}:{hi})", dev_state[i, lo:hi].cpu().numpy(),
                          host_state[i, lo:hi])


def run_workload(name, steps=None, sample_rows=64):
    w = synth.WORKLOADS[name]
    steps = w.steps if steps is None else steps
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    gen = synth.Generator.for_workload(w)
    gdt = torch.int16 if w.grad_dtype == "bf16" else torch.float32
    log(f"[workload] {name}: d={w.d} N={w.N} n={w.n} m={w.m} grad={w.grad_dtype} steps={steps}"
        f"{' tensors=%d' % len(w.views) if w.per_tensor else ''}")
    grad = torch.empty((w.N, w.d), dtype=gdt, device=dev)
    h = torch.zeros((w.N, w.d), dtype=torch.float32, device=dev)
    g = torch.zeros((w.N, w.d), dtype=torch.float32, device=dev)
    h_o = np.zeros((w.N, w.d), F32)
    g_o = np.zeros((w.N, w.d), F32)
    buckets = w.buckets()
    tensors = w.tensor_views() if w.per_tensor else None
    span = _row_spans(w)
    comp = arc.Compressor(d=w.d, N=w.N, n=w.n, r=w.r, K=w.K_global(), eta=w.eta,
                          seed=w.sketch_seed, grad_dtype=w.grad_dtype, buckets=buckets,
                          tensors=tensors, device=dev, stream=stream)
    log(f"[workload] {name}: {comp.describe()}")
    rng = np.random.default_rng(12345)
    try:
        for t in range(steps):
            with timed(f"{name} t={t} generate+copy"):
                gen.fill_device(t, grad, stream)
                grad_np = _host_copy(grad)
            with timed(f"{name} t={t} gpu step"):
                idx, agg = comp.step(t, grad, h, g)
                sigma = comp.sigma()
                torch.cuda.synchronize(dev)
            with timed(f"{name} t={t} oracle step ({oracle.num_threads()} threads)"):
                if tensors is None:
                    want = oracle.step(h_o, g_o, grad_np, n=w.n, r=w.r, eta=w.eta,
                                       seed=w.sketch_seed, t=t, K=w.K_global(),
                                       buckets=buckets, want_sigma=True)
                else:
                    want = oracle.step_tensors(h_o, g_o, grad_np, tensors, r=w.r, eta=w.eta,
                                               seed=w.sketch_seed, t=t, want_sigma=True)
            del grad_np
            got_idx = idx.cpu().numpy()
            assert np.array_equal(got_idx, want["idx"]), f"{name} t={t}: selected rows differ"
            compare_float(f"{name} t={t} sigma", sigma.cpu().numpy(), want["sigma"])
            compare_float(f"{name} t={t} agg", agg.cpu().numpy(), want["agg"])
            rows = np.unique(np.concatenate([
                rng.choice(w.m, size=min(sample_rows, w.m), replace=False),
                got_idx[rng.choice(len(got_idx), size=min(sample_rows, len(got_idx)),
                                   replace=False)] if len(got_idx) else np.zeros(0, int),
                [w.m - 1]]))
            _compare_rows(f"{name} t={t} h", h, h_o, rows, span)
            _compare_rows(f"{name} t={t} g", g, g_o, rows, span)
            log(f"[workload] {name} t={t}: {len(got_idx)} rows bit-exact; sampled "
                f"{len(rows)} rows of h, g bit-exact")
        with timed(f"{name} full state compare"):
            _compare_full(f"{name} final h", h, h_o)
            _compare_full(f"{name} final g", g, g_o)
        log(f"[workload] {name}: final h and g bit-exact over all {w.N * w.d} elements")
    finally:
        comp.close()


@pytest.mark.timeout(300)
def test_workload_tiny():
    run_workload("tiny")


@pytest.mark.timeout(600)
def test_workload_resnet18():
    run_workload("resnet18")


@pytest.mark.timeout(600)
def test_workload_gpt2s():
    run_workload("gpt2s")


@pytest.mark.timeout(900)
def test_workload_llama1b():
    run_workload("llama1b")


@pytest.mark.timeout(600)
def test_workload_resnet18_per_tensor():
    run_workload("resnet18_tensors")


@pytest.mark.timeout(600)
def test_workload_gpt2s_per_tensor():
    run_workload("gpt2s_tensors")


@pytest.mark.timeout(900)
def test_workload_llama1b_per_tensor():
    run_workload("llama1b_tensors")


@pytest.mark.timeout(1200)
@pytest.mark.skipif(os.environ.get("ARC_SKIP_LLAMA7B") == "1",
                    reason="ARC_SKIP_LLAMA7B=1 (needs ~140 GB host RAM and ~140 GB HBM)")
def test_workload_llama7b_buckets():
    run_workload("llama7b")
