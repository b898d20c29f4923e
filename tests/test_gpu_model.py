"""GPU parity of the model step around the compressor (arc_model_step):
dense warm-up iterations, then compressed ones, with the SGD (Eq. (11c)),
heavy-ball and Adam updates, against the oracle's dense step, compressor
step, G accumulation and optimiser.  Every state array is compared bit for
bit after every iteration."""
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


def run_model_case(*, d, N, n=0, tensors=None, r=4, K=0, eta=0.1, seed=3, grad_dtype="f32",
                   family=0, optimizer="adam", steps=4, dense_steps=1, lr=1e-2, momentum=0.9,
                   beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0, misalign=0,
                   compressor="arc", label="model"):
    dev = torch.device("cuda:0")
    sizes = None if tensors is None else [a * b for a, b, _ in tensors]
    gen = synth.Generator(d, N, 21, grad_dtype=grad_dtype, family=family, tensors=sizes)
    mc = arc.make_model_config(optimizer, lr=lr, dense_steps=dense_steps, momentum=momentum,
                               beta1=beta1, beta2=beta2, eps=eps, weight_decay=weight_decay)
    comp = arc.Compressor(d=d, N=N, n=n, r=r, K=K, eta=eta, seed=seed, grad_dtype=grad_dtype,
                          tensors=tensors, compressor=compressor, device=dev)
    try:
        h = device_buffer((N, d), torch.float32, dev, misalign)
        g = device_buffer((N, d), torch.float32, dev, misalign)
        G = device_buffer((d,), torch.float32, dev, misalign)
        x = device_buffer((d,), torch.float32, dev, misalign)
        m = device_buffer((d,), torch.float32, dev, misalign)
        v = device_buffer((d,), torch.float32, dev, misalign)
        rng = np.random.default_rng(8)
        x0 = rng.standard_normal(d).astype(F32)
        x.copy_(torch.from_numpy(x0))
        h_o, g_o = np.zeros((N, d), F32), np.zeros((N, d), F32)
        G_o, x_o, m_o, v_o = np.zeros(d, F32), x0.copy(), np.zeros(d, F32), np.zeros(d, F32)
        for t in range(steps):
            grad_np = gen.fill_host(t)
            grad = to_device_grad(grad_np, dev)
            if misalign:
                gbuf = torch.zeros(grad.numel() + misalign, dtype=grad.dtype, device=dev)
                gbuf[misalign:].copy_(grad.view(-1))
                grad = gbuf[misalign:].view(N, d)
            idx, agg = comp.model_step(t, grad, h, g, G, x, mc, m, v)
            torch.cuda.synchronize(dev)
            if t < dense_steps:
                oracle.dense_step(h_o, g_o, G_o, grad_np, eta)
            elif compressor == "randk":
                if tensors is None:
                    want = oracle.step_randk(h_o, g_o, grad_np, eta=eta, seed=seed, t=t, n=n, K=K)
                    oracle.accumulate(G_o, want["idx"], want["agg"], n=n)
                else:
                    want = oracle.step_randk(h_o, g_o, grad_np, eta=eta, seed=seed, t=t,
                                             tensors=tensors)
                    oracle.accumulate(G_o, want["idx"], want["agg"], tensors=tensors)
                assert np.array_equal(idx.cpu().numpy(), want["idx"]), f"{label} t={t} idx"
                compare_float(f"{label} t={t} agg", agg.cpu().numpy().reshape(-1),
                              want["agg"].reshape(-1))
            elif compressor == "topk":
                if tensors is None:
                    want = oracle.step_topk(h_o, g_o, grad_np, eta=eta, n=n, K=K)
                    oracle.merge_topk(G_o, want["idx"], want["agg"], n=n)
                else:
                    want = oracle.step_topk(h_o, g_o, grad_np, eta=eta, tensors=tensors)
                    oracle.merge_topk(G_o, want["idx"], want["agg"], tensors=tensors)
                assert np.array_equal(idx.cpu().numpy(), want["idx"]), f"{label} t={t} idx"
                compare_float(f"{label} t={t} agg", agg.cpu().numpy().reshape(-1),
                              want["agg"].reshape(-1))
            else:
                if tensors is None:
                    want = oracle.step(h_o, g_o, grad_np, n=n, r=r, eta=eta, seed=seed, t=t, K=K)
                    oracle.accumulate(G_o, want["idx"], want["agg"], n=n)
                else:
                    want = oracle.step_tensors(h_o, g_o, grad_np, tensors, r=r, eta=eta,
                                               seed=seed, t=t)
                    oracle.accumulate(G_o, want["idx"], want["agg"], tensors=tensors)
                assert np.array_equal(idx.cpu().numpy(), want["idx"]), f"{label} t={t} idx"
                compare_float(f"{label} t={t} agg", agg.cpu().numpy().reshape(-1),
                              want["agg"].reshape(-1))
            oracle.optimizer_step(optimizer, G_o, x_o, m_o, v_o, N=N, T=t + 1, lr=lr,
                                  momentum=momentum, beta1=beta1, beta2=beta2, eps=eps,
                                  weight_decay=weight_decay)
            for name, dv, hv in (("h", h, h_o), ("g", g, g_o), ("G", G, G_o), ("x", x, x_o)):
                compare_float(f"{label} t={t} {name}", dv.cpu().numpy(), hv)
            if optimizer != "sgd":
                compare_float(f"{label} t={t} m", m.cpu().numpy(), m_o)
            if optimizer == "adam":
                compare_float(f"{label} t={t} v", v.cpu().numpy(), v_o)
    finally:
        comp.close()


MIXED = [(70, 147, 9), (1, 64, 1), (129, 64, 4), (40, 512, 3), (2, 2, 2)]
PARTIAL = [(70, 100, 9), (1, 1000, 1), (33, 36, 3), (5, 4, 2), (129, 200, 4)]

CASES = [
    ("sgd_f32", dict(d=256 * 300, N=4, n=256, K=9, optimizer="sgd", lr=0.5)),
    ("msgd_bf16", dict(d=512 * 200 + 8, N=3, n=512, K=5, optimizer="msgd", grad_dtype="bf16",
                       family=1, momentum=0.9)),
    ("adam_f32_wd", dict(d=768 * 100, N=8, n=768, K=7, optimizer="adam", weight_decay=5e-4)),
    ("adam_bf16_dense2", dict(d=2048 * 40, N=4, n=2048, K=3, optimizer="adam",
                              grad_dtype="bf16", family=1, dense_steps=2, steps=5)),
    ("adam_general_n100", dict(d=100 * 321 + 7, N=3, n=100, r=3, K=12, optimizer="adam")),
    ("adam_tensors", dict(d=sum(a * b for a, b, _ in MIXED), N=3, tensors=MIXED,
                          optimizer="adam")),
    ("sgd_all_dense", dict(d=4096 + 12, N=2, n=64, K=3, optimizer="sgd", dense_steps=10,
                           steps=3)),
    ("msgd_no_dense", dict(d=256 * 64, N=5, n=256, K=4, optimizer="msgd", dense_steps=0)),
    ("adam_per_worker_N12", dict(d=256 * 100, N=12, n=256, K=6, optimizer="adam")),
    ("msgd_partial_chunk_tensors", dict(d=sum(a * b for a, b, _ in PARTIAL), N=4,
                                        tensors=PARTIAL, optimizer="msgd")),
    # Top-K: each node's own rows, merged into G in ascending node order
    ("topk_sgd_f32", dict(d=256 * 300, N=4, n=256, K=9, optimizer="sgd", lr=0.5,
                          compressor="topk")),
    ("topk_adam_bf16_ragged", dict(d=512 * 200 + 8, N=3, n=512, K=20, optimizer="adam",
                                   grad_dtype="bf16", family=1, compressor="topk")),
    ("topk_msgd_many_blocks", dict(d=32 * 20000, N=2, n=32, K=3000, optimizer="msgd",
                                   compressor="topk", steps=3)),
    ("topk_adam_tensors", dict(d=sum(a * b for a, b, _ in MIXED), N=3, tensors=MIXED,
                               optimizer="adam", compressor="topk")),
    ("topk_keep_all", dict(d=64 * 50 + 12, N=5, n=64, K=51, optimizer="sgd",
                           compressor="topk", dense_steps=0)),
    ("topk_partial_tensors_N8", dict(d=sum(a * b for a, b, _ in PARTIAL), N=8,
                                     tensors=PARTIAL, optimizer="adam", compressor="topk")),
    ("topk_general_n100", dict(d=100 * 321 + 7, N=3, n=100, K=12, optimizer="adam",
                               compressor="topk")),
]


@pytest.mark.parametrize("name,kw", CASES, ids=[c[0] for c in CASES])
def test_model_step_parity(name, kw):
    log(f"[model] {name} {kw if 'tensors' not in kw else '(tensors)'}")
    run_model_case(label=name, **kw)


@pytest.mark.parametrize("compressor", ["arc", "topk"])
def test_model_step_misaligned_pointers(compressor):
    log(f"[model] misaligned {compressor}")
    run_model_case(label=f"model_misaligned_{compressor}", d=256 * 80, N=3, n=256, K=5,
                   optimizer="adam", misalign=1, dense_steps=1, steps=3, compressor=compressor)


def test_model_step_rejects_bad_settings():
    d, N = 256 * 10, 2
    comp = arc.Compressor(d=d, N=N, n=256, K=2, eta=0.1, seed=5)
    try:
        z = lambda *s: torch.zeros(*s, device="cuda")  # noqa: E731
        grad, h, g = z((N, d)), z((N, d)), z((N, d))
        G, x, m, v = z(d), z(d), z(d), z(d)
        bad = [
            (arc.make_model_config("adam", lr=0.1), dict(v=None), "opt_v"),
            (arc.make_model_config("msgd", lr=0.1), dict(m=None), "opt_m"),
            (arc.make_model_config("sgd", lr=float("inf")), {}, "finite"),
            (arc.make_model_config("adam", lr=0.1, beta1=1.0), {}, "beta"),
            (arc.make_model_config("sgd", lr=0.1, dense_steps=-1), {}, "dense_steps"),
            (arc.make_model_config(7, lr=0.1), {}, "optimizer"),
            (arc.make_model_config("sgd", lr=0.1), dict(x=G), "overlap"),
            (arc.make_model_config("sgd", lr=0.1), dict(G=h[0]), "overlap"),
        ]
        for mc, repl, msg in bad:
            args = dict(G=G, x=x, m=m, v=v)
            args.update(repl)
            with pytest.raises(arc.ArcError, match=msg):
                arc.arc_model_step(comp.ctx, mc, 0, grad, h, g, args["G"], args["x"], args["m"],
                                   args["v"], comp.idx, comp.agg)
        # a dense iteration needs no output buffers
        mc = arc.make_model_config("sgd", lr=0.1, dense_steps=1)
        arc.arc_model_step(comp.ctx, mc, 0, grad, h, g, G, x, None, None, None, None)
        torch.cuda.synchronize()
    finally:
        comp.close()


@pytest.mark.timeout(900)
def test_model_step_full_size_llama1b_adam():
    """The 1.1B workload: one dense iteration, then two compressed ones, with
    Adam and weight decay; every state array compared in full."""
    w = synth.WORKLOADS["llama1b"]
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    gen = synth.Generator.for_workload(w)
    mc = arc.make_model_config("adam", lr=1e-3, dense_steps=1, weight_decay=5e-4)
    comp = arc.Compressor(d=w.d, N=w.N, n=w.n, r=w.r, K=w.K_global(), eta=w.eta,
                          seed=w.sketch_seed, grad_dtype=w.grad_dtype, device=dev, stream=stream)
    try:
        grad = torch.empty((w.N, w.d), dtype=torch.int16, device=dev)
        h = torch.zeros((w.N, w.d), device=dev)
        g = torch.zeros((w.N, w.d), device=dev)
        G, x, m, v = (torch.zeros(w.d, device=dev) for _ in range(4))
        h_o, g_o = np.zeros((w.N, w.d), F32), np.zeros((w.N, w.d), F32)
        G_o, x_o, m_o, v_o = (np.zeros(w.d, F32) for _ in range(4))
        for t in range(3):
            gen.fill_device(t, grad, stream)
            grad_np = grad.cpu().numpy().view(np.uint16)
            idx, agg = comp.model_step(t, grad, h, g, G, x, mc, m, v)
            torch.cuda.synchronize(dev)
            if t < 1:
                oracle.dense_step(h_o, g_o, G_o, grad_np, w.eta)
            else:
                want = oracle.step(h_o, g_o, grad_np, n=w.n, r=w.r, eta=w.eta,
                                   seed=w.sketch_seed, t=t, K=w.K_global())
                oracle.accumulate(G_o, want["idx"], want["agg"], n=w.n)
                assert np.array_equal(idx.cpu().numpy(), want["idx"]), t
                compare_float(f"llama1b model t={t} agg", agg.cpu().numpy(), want["agg"])
            del grad_np
            oracle.optimizer_step("adam", G_o, x_o, m_o, v_o, N=w.N, T=t + 1, lr=1e-3,
                                  weight_decay=5e-4)
            for name, dv, hv in (("G", G, G_o), ("x", x, x_o), ("m", m, m_o), ("v", v, v_o)):
                compare_float(f"llama1b model t={t} {name}", dv.cpu().numpy(), hv)
            log(f"[model] llama1b t={t}: G, x, m, v bit-exact over {w.d} coordinates")
        for i in range(w.N):
            compare_float(f"llama1b model h[{i}]", h[i].cpu().numpy(), h_o[i])
            compare_float(f"llama1b model g[{i}]", g[i].cpu().numpy(), g_o[i])
    finally:
        comp.close()


@pytest.mark.timeout(900)
def test_model_step_full_size_gpt2s_topk_adam():
    """The GPT-2-small workload with Top-K in the model step: every node's own
    163 rows, merged into G over the 8 nodes; two compressed iterations with
    Adam, G, x, m, v, h and g compared in full."""
    w = synth.WORKLOADS["gpt2s"]
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    gen = synth.Generator.for_workload(w)
    mc = arc.make_model_config("adam", lr=1e-3, dense_steps=0, weight_decay=5e-4)
    comp = arc.Compressor(d=w.d, N=w.N, n=w.n, r=w.r, K=w.K_global(), eta=w.eta,
                          seed=w.sketch_seed, compressor="topk", device=dev, stream=stream)
    try:
        grad = torch.empty((w.N, w.d), dtype=torch.float32, device=dev)
        h = torch.zeros((w.N, w.d), device=dev)
        g = torch.zeros((w.N, w.d), device=dev)
        G, x, m, v = (torch.zeros(w.d, device=dev) for _ in range(4))
        h_o, g_o = np.zeros((w.N, w.d), F32), np.zeros((w.N, w.d), F32)
        G_o, x_o, m_o, v_o = (np.zeros(w.d, F32) for _ in range(4))
        for t in range(2):
            gen.fill_device(t, grad, stream)
            grad_np = grad.cpu().numpy()
            idx, agg = comp.model_step(t, grad, h, g, G, x, mc, m, v)
            torch.cuda.synchronize(dev)
            want = oracle.step_topk(h_o, g_o, grad_np, eta=w.eta, n=w.n, K=w.K_global())
            oracle.merge_topk(G_o, want["idx"], want["agg"], n=w.n)
            assert np.array_equal(idx.cpu().numpy(), want["idx"]), t
            compare_float(f"gpt2s topk model t={t} agg", agg.cpu().numpy().reshape(-1),
                          want["agg"].reshape(-1))
            del grad_np
            oracle.optimizer_step("adam", G_o, x_o, m_o, v_o, N=w.N, T=t + 1, lr=1e-3,
                                  weight_decay=5e-4)
            for name, dv, hv in (("G", G, G_o), ("x", x, x_o), ("m", m, m_o), ("v", v, v_o)):
                compare_float(f"gpt2s topk model t={t} {name}", dv.cpu().numpy(), hv)
            log(f"[model] gpt2s topk t={t}: G, x, m, v bit-exact over {w.d} coordinates")
        for i in range(w.N):
            compare_float(f"gpt2s topk model h[{i}]", h[i].cpu().numpy(), h_o[i])
            compare_float(f"gpt2s topk model g[{i}]", g[i].cpu().numpy(), g_o[i])
    finally:
        comp.close()
