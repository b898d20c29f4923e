"""Helpers for the GPU parity tests: run libarctopk and the CPU oracle on the
same seeded inputs, step by step, and compare.

The bar: selected rows and the importance Sigma bit-exact; agg, h and g within
1e-5 relative max-norm (and, with the canonical operation order both sides
follow, bit-exact as well).
"""
from __future__ import annotations

import sys
import time

import numpy as np
import torch

import oracle
import paper_2510_26709_amd as arc
import synth

F32 = np.float32
TOL = 1e-5


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def rel_max_err(got: np.ndarray, want: np.ndarray) -> float:
    if want.size == 0:
        return 0.0
    g64 = got.astype(np.float64)
    w64 = want.astype(np.float64)
    den = float(np.max(np.abs(w64)))
    num = float(np.max(np.abs(g64 - w64)))
    if den == 0.0:
        return 0.0 if num == 0.0 else float("inf")
    return num / den


def compare_float(name: str, got: np.ndarray, want: np.ndarray, bit_exact: bool = True) -> None:
    assert got.shape == want.shape, (name, got.shape, want.shape)
    if np.array_equal(got.view(np.uint32), want.view(np.uint32)):
        return  # bit-exact, hence also within the tolerance
    err = rel_max_err(got, want)
    assert err <= TOL, f"{name}: relative max-norm error {err:.3e} > {TOL}"
    if bit_exact:
        diff = got.view(np.uint32) != want.view(np.uint32)
        if np.any(diff):
            first = np.argwhere(diff)[0]
            raise AssertionError(
                f"{name}: {int(diff.sum())} elements differ in bits (rel err {err:.3e}); "
                f"first at {tuple(first)}: {got[tuple(first)]!r} vs {want[tuple(first)]!r}")


def to_device_grad(grad_np: np.ndarray, dev) -> torch.Tensor:
    if grad_np.dtype == np.uint16:
        return torch.from_numpy(grad_np.view(np.int16)).to(dev)
    return torch.from_numpy(grad_np).to(dev)


def device_buffer(shape, dtype, dev, misalign_floats: int = 0) -> torch.Tensor:
    """Zeroed device tensor; misalign_floats > 0 offsets its start by that many
    elements from a 256-byte aligned allocation."""
    numel = int(np.prod(shape))
    base = torch.zeros(numel + misalign_floats, dtype=dtype, device=dev)
    return base[misalign_floats:].view(*shape)


def run_case(*, d, N, n=0, r=4, K=0, eta=0.1, seed=7, grad_dtype="f32", buckets=None,
             tensors=None, steps=2, grad_fn=None, data_seed=11, family=0, V=None, misalign=0,
             check_S=False, bit_exact=True, dev="cuda:0", label="case", ts=None):
    """Run `steps` steps of libarctopk and of the oracle from h = g = 0
    (step numbers 0, 1, ..., or the sequence ts).
    tensors = [(rows, cols, K), ...] selects the per-tensor mode."""
    dev = torch.device(dev)
    gen = None
    if grad_fn is None:
        sizes = None if tensors is None else [a * b for a, b, _ in tensors]
        gen = synth.Generator(d, N, data_seed, grad_dtype=grad_dtype, family=family,
                              tensors=sizes)
        grad_fn = gen.fill_host
    comp = arc.Compressor(d=d, N=N, n=n, r=r, K=K, eta=eta, seed=seed, grad_dtype=grad_dtype,
                          buckets=buckets, tensors=tensors, device=dev)
    try:
        if V is not None:
            arc.arc_set_projection(comp.ctx, np.ascontiguousarray(V, dtype=F32))
        h = device_buffer((N, d), torch.float32, dev, misalign)
        g = device_buffer((N, d), torch.float32, dev, misalign)
        h_o = np.zeros((N, d), F32)
        g_o = np.zeros((N, d), F32)
        for t in (range(steps) if ts is None else ts):
            grad_np = grad_fn(t)
            grad = to_device_grad(grad_np, dev)
            if misalign:
                gbuf = torch.zeros(grad.numel() + misalign, dtype=grad.dtype, device=dev)
                gbuf[misalign:].copy_(grad.view(-1))
                grad = gbuf[misalign:].view(N, d)
            idx, agg = comp.step(t, grad, h, g)
            sigma = comp.sigma()
            S = comp.sketch() if check_S else None
            torch.cuda.synchronize(dev)
            if tensors is None:
                want = oracle.step(h_o, g_o, grad_np, n=n, r=r, eta=eta, seed=seed, t=t, K=K,
                                   buckets=buckets, V=V, want_sigma=True, want_S=check_S)
            else:
                want = oracle.step_tensors(h_o, g_o, grad_np, tensors, r=r, eta=eta, seed=seed,
                                           t=t, want_sigma=True, want_S=check_S)
            got_idx = idx.cpu().numpy()
            assert np.array_equal(got_idx, want["idx"]), \
                f"{label} t={t}: selected rows differ: {got_idx[:10]} vs {want['idx'][:10]}"
            compare_float(f"{label} t={t} sigma", sigma.cpu().numpy(), want["sigma"], True)
            if check_S:
                compare_float(f"{label} t={t} S", S.cpu().numpy(), want["S"], True)
            compare_float(f"{label} t={t} agg", agg.cpu().numpy(), want["agg"], bit_exact)
            compare_float(f"{label} t={t} h", h.cpu().numpy(), h_o, bit_exact)
            compare_float(f"{label} t={t} g", g.cpu().numpy(), g_o, bit_exact)
        return comp.K_total
    finally:
        comp.close()


def timed(label):
    class _T:
        def __enter__(self):
            self.t0 = time.time()
            return self

        def __exit__(self, *a):
            log(f"  {label}: {time.time() - self.t0:.2f}s")
    return _T()
