"""GPU parity of the per-tensor mode against the CPU oracle: each tensor in its
own 2-D view with its own K (Table I's setting; Sec. VI compresses matrices
and reshaped convolution kernels, 1-D tensors whole).  The layouts cover full
and partial 64-row groups, widths that are and are not multiples of 32,
tensor offsets that break 16-byte alignment, one-row tensors, K = 0,
K >= rows, shared projections (equal widths), and the general kernels."""
import numpy as np
import pytest
import torch

import paper_2510_26709_amd as arc
from parity_util import log, run_case

pytestmark = pytest.mark.gpu
F32 = np.float32


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _d(tensors):
    return sum(r * c for r, c, _ in tensors)


# Every tensor 16-byte aligned, widths multiples of 32: the vector kernels
# (groups of 64 rows and partial groups); equal widths share V.
ALIGNED = [(200, 96, 7), (1, 96, 1), (130, 256, 10), (64, 64, 64), (5, 32, 0), (1, 64, 1),
           (100, 512, 3), (64, 96, 2)]
# Width 147 moves every later tensor off 16-byte alignment until an offset
# lands on a multiple of 4 again; widths 33 and 7 are never vectorisable.
MIXED = [(70, 147, 9), (3, 33, 1), (64, 96, 5), (1, 7, 1), (129, 64, 4), (1, 64, 1),
         (77, 160, 77), (2, 2, 5)]

# Widths that are multiples of 4 but not of any chunk width: vector groups
# whose rows end in a partial chunk (16-, 32- and 64-row groups).
PARTIAL = [(70, 100, 9), (1, 1000, 1), (33, 36, 3), (5, 4, 2), (129, 200, 4), (2, 520, 1),
           (64, 96, 5), (300, 44, 11)]

# Wide rows: 16-row groups of 2048 columns and 32-row groups of 576 (16 and 9
# chunks) take workgroups of two waves, one per compute unit, while the
# 8-row groups (768, 3072 and 4096 columns: 8.7 chunks on average) take
# workgroups of four, one per compute unit, in a launch beside them.  The
# first 64 rows of the 2048-wide tensor and the first 32 of the 3072-wide
# one form groups of every 4th row.
WIDE = [(70, 2048, 3), (100, 768, 5), (40, 3072, 2), (1, 4096, 1), (64, 576, 4)]


def _random_layout(seed, count, max_rows=300):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(count):
        if rng.random() < 0.3:
            out.append((1, int(rng.integers(1, 700)), 1))
        else:
            rows = int(rng.integers(1, max_rows))
            cols = int(rng.choice([32, 64, 96, 128, 160, 256, 40, 100, 147]))
            out.append((rows, cols, int(rng.integers(0, rows + 2))))
    d = sum(r * c for r, c, _ in out)
    if d % 4:
        out.append((1, 4 - d % 4, 1))  # d % 4 == 0: vectorisable tensors stay so
    return out


CASES = [
    ("aligned_f32_N3", dict(tensors=ALIGNED, N=3, r=4, steps=3)),
    ("aligned_bf16_N4", dict(tensors=ALIGNED, N=4, r=4, steps=2, grad_dtype="bf16", family=1)),
    ("aligned_r2_N2", dict(tensors=ALIGNED, N=2, r=2, steps=2)),
    ("aligned_r8_N5", dict(tensors=ALIGNED, N=5, r=8, steps=2)),
    ("aligned_r1_N8", dict(tensors=ALIGNED, N=8, r=1, steps=2)),
    ("aligned_per_worker_N10", dict(tensors=ALIGNED, N=10, r=4, steps=2)),
    ("aligned_bf16_per_worker_N9", dict(tensors=ALIGNED, N=9, r=4, steps=2, grad_dtype="bf16",
                                        family=1)),
    ("mixed_f32_N3", dict(tensors=MIXED, N=3, r=4, steps=3)),
    ("mixed_bf16_N2", dict(tensors=MIXED, N=2, r=4, steps=2, grad_dtype="bf16", family=1)),
    ("mixed_r3_general", dict(tensors=MIXED, N=3, r=3, steps=2)),
    ("mixed_per_worker_N12", dict(tensors=MIXED, N=12, r=4, steps=2)),
    ("partial_f32_N3", dict(tensors=PARTIAL, N=3, r=4, steps=3)),
    ("partial_bf16_per_worker_N4", dict(tensors=PARTIAL, N=4, r=4, steps=2, grad_dtype="bf16",
                                        family=1)),
    ("partial_r8_N2", dict(tensors=PARTIAL, N=2, r=8, steps=2)),
    ("partial_r1_bf16_N7", dict(tensors=PARTIAL, N=7, r=1, steps=2, grad_dtype="bf16", family=1)),
    ("wide_two_wave_bf16_N3", dict(tensors=WIDE, N=3, r=4, steps=2, grad_dtype="bf16", family=1)),
    ("wide_two_wave_r1_N2", dict(tensors=WIDE, N=2, r=1, steps=2)),
    ("one_tensor_multiblock_select", dict(tensors=[(40_000, 32, 9_000)], N=2, r=4, steps=2)),
    ("single_one_row_tensor", dict(tensors=[(1, 4096, 1)], N=2, r=4, steps=2)),
    ("all_k_zero", dict(tensors=[(64, 64, 0), (10, 32, 0)], N=2, r=4, steps=2)),
    ("random_layout_60", dict(tensors=_random_layout(3, 60), N=4, r=4, steps=2)),
    ("random_layout_250_bf16", dict(tensors=_random_layout(4, 250, 120), N=3, r=4, steps=2,
                                    grad_dtype="bf16", family=1)),
]


@pytest.mark.parametrize("name,kw", CASES, ids=[c[0] for c in CASES])
def test_tensor_parity(name, kw):
    kw = dict(kw)
    kw["d"] = _d(kw["tensors"])
    log(f"[tensors] {name} d={kw['d']} tensors={len(kw['tensors'])} N={kw['N']} r={kw['r']}")
    run_case(label=name, check_S=True, **kw)


def test_tensor_parity_misaligned_pointers():
    log("[tensors] misaligned")
    run_case(label="tensors_misaligned", d=_d(ALIGNED), N=3, r=4, tensors=ALIGNED, steps=2,
             misalign=1, check_S=True)
    # groups of rows 4 apart, taken by the general kernel
    log("[tensors] misaligned wide")
    run_case(label="tensors_misaligned_wide", d=_d(WIDE), N=2, r=4, tensors=WIDE, steps=1,
             misalign=1, check_S=True)


def test_tensor_parity_zero_residual_ties():
    d = _d(ALIGNED)
    zero = np.zeros((2, d), F32)
    log("[tensors] zero residual")
    run_case(label="tensors_zeros", d=d, N=2, r=4, tensors=ALIGNED, steps=2,
             grad_fn=lambda t: zero)


def test_tensor_mode_launch_shapes():
    comp = arc.Compressor(d=_d(WIDE), N=2, r=4, tensors=WIDE, eta=0.1, seed=1)
    try:
        desc = comp.describe()
        assert "workgroup_waves=(4 2/cu 2/cu 4/cu) interleaved_groups=8 " in desc, desc
    finally:
        comp.close()


def test_tensor_mode_describe_and_payload():
    comp = arc.Compressor(d=_d(MIXED), N=3, r=4, tensors=MIXED, eta=0.1, seed=1)
    try:
        desc = comp.describe()
        log(f"[describe] {desc}")
        assert "mode=tensors" in desc
        # 147, 33, 96, 7, 64, 160, 2: distinct widths
        assert "widths=7 " in desc
        kept = [min(k, r) for r, _, k in MIXED]
        assert comp.K_total == sum(kept)
        assert comp.payload == sum(k * c for k, (_, c, _) in zip(kept, MIXED))
        assert comp.m == sum(r for r, _, _ in MIXED)
    finally:
        comp.close()


def test_tensor_mode_rejects_single_view_hooks():
    comp = arc.Compressor(d=_d(ALIGNED), N=2, r=4, tensors=ALIGNED, eta=0.1, seed=1)
    try:
        with pytest.raises(arc.ArcError, match="ARC_ERR_UNSUPPORTED"):
            arc.arc_set_projection(comp.ctx, np.ones((96, 4), F32))
        with pytest.raises(arc.ArcError, match="ARC_ERR_UNSUPPORTED"):
            arc.arc_debug_projection(comp.ctx, 0, np.empty((96, 4), F32))
    finally:
        comp.close()


def test_single_view_equals_per_tensor_with_one_tensor():
    """A single m x n view with d = m*n and one tensor (m, n, K) are the same
    compressor: identical outputs, bit for bit."""
    m, n, K, N = 3000, 128, 37, 3
    d = m * n
    outs = []
    for tensors in (None, [(m, n, K)]):
        comp = arc.Compressor(d=d, N=N, n=0 if tensors else n, r=4, K=0 if tensors else K,
                              eta=0.1, seed=9, tensors=tensors)
        gen = torch.Generator().manual_seed(5)
        grad = torch.randn((N, d), generator=gen).cuda()
        h = torch.zeros((N, d), device="cuda")
        g = torch.zeros((N, d), device="cuda")
        res = []
        for t in range(2):
            idx, agg = comp.step(t, grad, h, g)
            res.append((idx.cpu().numpy().copy(), agg.reshape(-1).cpu().numpy().copy()))
        torch.cuda.synchronize()
        outs.append((res, h.cpu().numpy(), g.cpu().numpy()))
        comp.close()
    (r0, h0, g0), (r1, h1, g1) = outs
    for (i0, a0), (i1, a1) in zip(r0, r1):
        assert np.array_equal(i0, i1)
        assert a0.tobytes() == a1.tobytes()
    assert h0.tobytes() == h1.tobytes() and g0.tobytes() == g1.tobytes()
