"""GPU parity of the comparison compressors of Table I (Rand-K, Top-K) in the
same EF21M step, against the oracle's Rand-K and Top-K steps: selected rows
bit-exact, payload, h and g bit-exact, on single views (vectorised, general,
ragged, buckets, bf16) and per-tensor layouts, and at full size."""
import numpy as np
import pytest
import torch

import oracle
import paper_2510_26709_amd as arc
import synth
from parity_util import compare_float, device_buffer, log, to_device_grad

pytestmark = pytest.mark.gpu
F32 = np.float32


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def run_compare_case(*, compressor, d, N, n=0, tensors=None, K=0, buckets=None, eta=0.1,
                     seed=17, grad_dtype="f32", family=0, steps=2, misalign=0, label="cmp"):
    dev = torch.device("cuda:0")
    sizes = None if tensors is None else [a * b for a, b, _ in tensors]
    gen = synth.Generator(d, N, 31, grad_dtype=grad_dtype, family=family, tensors=sizes)
    comp = arc.Compressor(d=d, N=N, n=n, K=K, eta=eta, seed=seed, grad_dtype=grad_dtype,
                          buckets=buckets, tensors=tensors, compressor=compressor, device=dev)
    try:
        h = device_buffer((N, d), torch.float32, dev, misalign)
        g = device_buffer((N, d), torch.float32, dev, misalign)
        h_o, g_o = np.zeros((N, d), F32), np.zeros((N, d), F32)
        for t in range(steps):
            grad_np = gen.fill_host(t)
            grad = to_device_grad(grad_np, dev)
            if misalign:
                gbuf = torch.zeros(grad.numel() + misalign, dtype=grad.dtype, device=dev)
                gbuf[misalign:].copy_(grad.view(-1))
                grad = gbuf[misalign:].view(N, d)
            idx, agg = comp.step(t, grad, h, g)
            torch.cuda.synchronize(dev)
            if compressor == "randk":
                want = oracle.step_randk(h_o, g_o, grad_np, eta=eta, seed=seed, t=t, n=n, K=K,
                                         buckets=buckets, tensors=tensors)
            else:
                want = oracle.step_topk(h_o, g_o, grad_np, eta=eta, n=n, K=K, buckets=buckets,
                                        tensors=tensors)
            got_idx = idx.cpu().numpy()
            assert np.array_equal(got_idx.reshape(want["idx"].shape), want["idx"]), \
                f"{label} t={t}: selected rows differ"
            compare_float(f"{label} t={t} agg", agg.cpu().numpy().reshape(-1),
                          want["agg"].reshape(-1))
            compare_float(f"{label} t={t} h", h.cpu().numpy(), h_o)
            compare_float(f"{label} t={t} g", g.cpu().numpy(), g_o)
        return comp.describe()
    finally:
        comp.close()


MIXED = [(70, 147, 9), (1, 64, 1), (129, 64, 4), (40, 512, 3), (2, 2, 2), (200, 96, 7)]
PARTIAL = [(70, 100, 9), (1, 1000, 1), (33, 36, 3), (5, 4, 2), (129, 200, 4), (64, 96, 5)]

CASES = [
    ("fast_f32_ragged", dict(d=256 * 700 + 40, N=3, n=256, K=9, steps=3)),
    ("fast_bf16", dict(d=512 * 300 + 8, N=4, n=512, K=5, grad_dtype="bf16", family=1)),
    ("generic_n100", dict(d=100 * 321 + 7, N=3, n=100, K=12)),
    ("buckets", dict(d=64 * 6000, N=3, n=64, buckets=([0, 1000, 1300, 1301, 5000, 6000],
                                                     [17, 500, 1, 0, 10]))),
    ("k_over", dict(d=256 * 50, N=2, n=256, K=10_000)),
    ("many_workers_N12", dict(d=256 * 300, N=12, n=256, K=7)),
    ("select_multiblock", dict(d=32 * 9000, N=2, n=32, K=2500)),
    ("tensors_mixed", dict(d=sum(a * b for a, b, _ in MIXED), N=3, tensors=MIXED)),
    ("tensors_bf16", dict(d=sum(a * b for a, b, _ in MIXED), N=2, tensors=MIXED,
                          grad_dtype="bf16", family=1)),
    ("partial_chunks_per_worker", dict(d=1000 * 60 + 996, N=5, n=1000, K=7)),
    ("two_wave_rows", dict(d=2304 * 120 + 36, N=3, n=2304, K=5, grad_dtype="bf16", family=1)),
    ("tensors_partial_bf16", dict(d=sum(a * b for a, b, _ in PARTIAL), N=3, tensors=PARTIAL,
                                  grad_dtype="bf16", family=1)),
]


@pytest.mark.parametrize("compressor", ["randk", "topk"])
@pytest.mark.parametrize("name,kw", CASES, ids=[c[0] for c in CASES])
def test_compare_parity(compressor, name, kw):
    log(f"[compare] {compressor} {name}")
    desc = run_compare_case(compressor=compressor, label=f"{compressor}_{name}", **kw)
    assert f"compressor={compressor}" in desc


@pytest.mark.parametrize("compressor", ["randk", "topk"])
def test_compare_misaligned(compressor):
    run_compare_case(compressor=compressor, d=256 * 120, N=3, n=256, K=11, misalign=1,
                     label=f"{compressor}_misaligned")


def test_randk_model_step():
    d, N, n, K = 256 * 64, 3, 256, 5
    dev = torch.device("cuda:0")
    mc = arc.make_model_config("sgd", lr=0.25, dense_steps=1)
    gen = synth.Generator(d, N, 5)
    comp = arc.Compressor(d=d, N=N, n=n, K=K, eta=0.1, seed=4, compressor="randk", device=dev)
    try:
        h, g = torch.zeros((N, d), device=dev), torch.zeros((N, d), device=dev)
        G, x = torch.zeros(d, device=dev), torch.zeros(d, device=dev)
        h_o, g_o = np.zeros((N, d), F32), np.zeros((N, d), F32)
        G_o, x_o = np.zeros(d, F32), np.zeros(d, F32)
        for t in range(3):
            grad_np = gen.fill_host(t)
            comp.model_step(t, torch.from_numpy(grad_np).to(dev), h, g, G, x, mc)
            torch.cuda.synchronize()
            if t < 1:
                oracle.dense_step(h_o, g_o, G_o, grad_np, 0.1)
            else:
                want = oracle.step_randk(h_o, g_o, grad_np, eta=0.1, seed=4, t=t, n=n, K=K)
                oracle.accumulate(G_o, want["idx"], want["agg"], n=n)
            oracle.optimizer_step("sgd", G_o, x_o, N=N, T=t + 1, lr=0.25)
            compare_float(f"randk model t={t} G", G.cpu().numpy(), G_o)
            compare_float(f"randk model t={t} x", x.cpu().numpy(), x_o)
    finally:
        comp.close()


@pytest.mark.timeout(900)
@pytest.mark.parametrize("compressor,name,steps", [("randk", "llama1b", 2),
                                                   ("topk", "llama1b", 2),
                                                   ("topk", "gpt2s_tensors", 2)])
def test_compare_full_size(compressor, name, steps):
    w = synth.WORKLOADS[name]
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    gen = synth.Generator.for_workload(w)
    tensors = w.tensor_views() if w.per_tensor else None
    gdt = torch.int16 if w.grad_dtype == "bf16" else torch.float32
    comp = arc.Compressor(d=w.d, N=w.N, n=w.n, r=w.r, K=w.K_global(), eta=w.eta,
                          seed=w.sketch_seed, grad_dtype=w.grad_dtype, buckets=w.buckets(),
                          tensors=tensors, compressor=compressor, device=dev, stream=stream)
    log(f"[compare] {compressor} {name}: {comp.describe()}")
    try:
        grad = torch.empty((w.N, w.d), dtype=gdt, device=dev)
        h = torch.zeros((w.N, w.d), device=dev)
        g = torch.zeros((w.N, w.d), device=dev)
        h_o, g_o = np.zeros((w.N, w.d), F32), np.zeros((w.N, w.d), F32)
        for t in range(steps):
            gen.fill_device(t, grad, stream)
            a = grad.cpu().numpy()
            grad_np = a.view(np.uint16) if a.dtype == np.int16 else a
            idx, agg = comp.step(t, grad, h, g)
            torch.cuda.synchronize(dev)
            kw = dict(n=w.n, K=w.K_global()) if tensors is None else dict(tensors=tensors)
            if compressor == "randk":
                want = oracle.step_randk(h_o, g_o, grad_np, eta=w.eta, seed=w.sketch_seed, t=t,
                                         **kw)
            else:
                want = oracle.step_topk(h_o, g_o, grad_np, eta=w.eta, **kw)
            del grad_np, a
            assert np.array_equal(idx.cpu().numpy().reshape(want["idx"].shape), want["idx"])
            compare_float(f"{compressor} {name} t={t} agg", agg.cpu().numpy().reshape(-1),
                          want["agg"].reshape(-1))
            log(f"[compare] {compressor} {name} t={t}: rows and payload bit-exact")
        for i in range(w.N):
            compare_float(f"{compressor} {name} h[{i}]", h[i].cpu().numpy(), h_o[i])
            compare_float(f"{compressor} {name} g[{i}]", g[i].cpu().numpy(), g_o[i])
    finally:
        comp.close()
