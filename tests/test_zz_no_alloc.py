"""The allocation-free entry point (arc_step_static) against arc_step: the
same configuration stepped through both on one stream from the same state,
every output compared bit for bit (selected rows, payload, h and g).  Calls
alternate between a larger and a smaller configuration, so that each call
finds the static device array holding the previous call's (different)
tables, sketch and selection state."""
import numpy as np
import pytest
import torch

import paper_2510_26709_amd as arc
import synth
from parity_util import compare_float, log, to_device_grad

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


class Pair:
    """One configuration run through arc_step (a context) and through
    arc_step_static, each with its own h and g."""

    def __init__(self, kw, stream, data_seed):
        self.kw = kw
        self.stream = stream
        self.N, self.d = kw["N"], kw["d"]
        grad_dtype = kw.get("grad_dtype", "f32")
        tensors = kw.get("tensors")
        sizes = None if tensors is None else [a * b for a, b, _ in tensors]
        self.gen = synth.Generator(self.d, self.N, data_seed, grad_dtype=grad_dtype,
                                   family=1 if grad_dtype == "bf16" else 0, tensors=sizes)
        self.comp = arc.Compressor(device=torch.device("cuda:0"), stream=stream, **kw)
        self.cfg, self.keep = arc.make_config(
            d=self.d, N=self.N, n=kw.get("n", 0), r=kw.get("r", 4), K=kw.get("K", 0),
            eta=kw["eta"], seed=kw["seed"],
            grad_dtype=arc.ARC_DTYPE_BF16 if grad_dtype == "bf16" else arc.ARC_DTYPE_F32,
            buckets=kw.get("buckets"), tensors=tensors, compressor=kw.get("compressor", "arc"))
        z = lambda: torch.zeros((self.N, self.d), dtype=torch.float32, device="cuda:0")
        self.h_ref, self.g_ref, self.h_st, self.g_st = z(), z(), z(), z()
        self.idx = torch.full((self.comp.K_total,), -1, dtype=torch.int32, device="cuda:0")
        self.agg = torch.full((self.comp.payload,), float("nan"), dtype=torch.float32,
                              device="cuda:0")

    def step_and_compare(self, t, label):
        log(f"[no-alloc] {label} t={t} d={self.d} N={self.N}")
        grad = to_device_grad(self.gen.fill_host(t), "cuda:0")
        with torch.cuda.stream(self.stream):
            idx_ref, agg_ref = self.comp.step(t, grad, self.h_ref, self.g_ref)
            arc.arc_step_static(self.cfg, self.stream, t, grad, self.h_st, self.g_st, self.idx,
                                self.agg)
        self.stream.synchronize()
        assert np.array_equal(self.idx.cpu().numpy(), idx_ref.reshape(-1).cpu().numpy()), label
        compare_float(f"{label} agg", self.agg.cpu().numpy(),
                      agg_ref.reshape(-1).cpu().numpy(), True)
        compare_float(f"{label} h", self.h_st.cpu().numpy(), self.h_ref.cpu().numpy(), True)
        compare_float(f"{label} g", self.g_st.cpu().numpy(), self.g_ref.cpu().numpy(), True)

    def close(self):
        self.comp.close()


BIG = dict(d=64 * 20000 + 32, N=3, n=64, r=4, K=700, eta=0.1, seed=31)  # 20,001 rows
SMALL = dict(d=256 * 300 + 8, N=2, n=256, r=4, K=9, eta=0.25, seed=32, grad_dtype="bf16")
TENSORS = dict(d=64 * 147 + 64 + 300 * 512 + 40 * 96, N=2, r=4, eta=0.1, seed=33,
               tensors=[(64, 147, 5), (1, 64, 1), (300, 512, 4), (40, 96, 40)])
BUCKETS = dict(d=128 * 9000, N=2, n=128, r=2, eta=0.1, seed=34,
               buckets=([0, 10, 8200, 9000], [3, 500, 800]))


def test_static_step_matches_arc_step_larger_then_smaller():
    stream = torch.cuda.Stream()
    big = Pair(BIG, stream, 101)
    small = Pair(SMALL, stream, 102)
    try:
        big.step_and_compare(0, "big")
        small.step_and_compare(0, "small")  # second call, smaller input
        big.step_and_compare(1, "big")
        small.step_and_compare(1, "small")
    finally:
        big.close()
        small.close()


def test_static_step_tensors_and_buckets():
    stream = torch.cuda.Stream()
    pairs = [Pair(TENSORS, stream, 103), Pair(BUCKETS, stream, 104)]
    try:
        for t in range(2):
            for p, label in zip(pairs, ("tensors", "buckets")):
                p.step_and_compare(t, label)
    finally:
        for p in pairs:
            p.close()


def test_static_step_comparison_compressors():
    # Rand-K (shared random rows) and Top-K (every node's own rows, over the
    # N*m row norms): the same static array, different scratch in it.
    stream = torch.cuda.Stream()
    pairs = [Pair(dict(BIG, compressor="topk"), stream, 105),
             Pair(dict(SMALL, compressor="randk"), stream, 106),
             Pair(dict(TENSORS, compressor="topk"), stream, 107)]
    try:
        for t in range(2):
            for p, label in zip(pairs, ("topk", "randk", "topk_tensors")):
                p.step_and_compare(t, label)
    finally:
        for p in pairs:
            p.close()


def test_static_step_gpt2s_full_size():
    # The GPT-2-small workload at full size: 20 MB of per-worker sketch in
    # the static array, multi-block selection over 162,031 rows.
    w = synth.WORKLOADS["gpt2s"]
    stream = torch.cuda.Stream()
    kw = dict(d=w.d, N=w.N, n=w.n, r=w.r, K=w.K_global(), eta=w.eta, seed=w.sketch_seed)
    comp = arc.Compressor(device=torch.device("cuda:0"), stream=stream, **kw)
    cfg, keep = arc.make_config(**kw)
    gen = synth.Generator.for_workload(w)
    try:
        grad = torch.empty((w.N, w.d), dtype=torch.float32, device="cuda:0")
        with torch.cuda.stream(stream):
            gen.fill_device(0, grad, stream)
            h_ref = torch.zeros_like(grad)
            g_ref = torch.zeros_like(grad)
            h_st = torch.zeros_like(grad)
            g_st = torch.zeros_like(grad)
            idx = torch.empty(comp.K_total, dtype=torch.int32, device="cuda:0")
            agg = torch.empty(comp.payload, dtype=torch.float32, device="cuda:0")
            for t in range(2):
                log(f"[no-alloc] gpt2s t={t}")
                idx_ref, agg_ref = comp.step(t, grad, h_ref, g_ref)
                arc.arc_step_static(cfg, stream, t, grad, h_st, g_st, idx, agg)
                stream.synchronize()
                assert torch.equal(idx, idx_ref)
                assert torch.equal(agg.view(torch.int32), agg_ref.reshape(-1).view(torch.int32))
                assert torch.equal(h_st.view(torch.int32), h_ref.view(torch.int32))
                assert torch.equal(g_st.view(torch.int32), g_ref.view(torch.int32))
    finally:
        comp.close()
