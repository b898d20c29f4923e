"""GPU parity of libarctopk against the CPU oracle on small seeded cases that
span several tiles, ragged tails, every kernel path and the degenerate cases
of the method (K = 0, K >= m, all-equal importance, buckets)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2510_26709_amd as arc
import synth
from parity_util import log, run_case

pytestmark = pytest.mark.gpu
F32 = np.float32


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


# name, kwargs.  "fast" = vectorised sketch (n % 32 == 0, d % 4 == 0, r in 1/2/4/8)
CASES = [
    ("fast_f32_ragged", dict(d=256 * 700 + 40, N=3, n=256, r=4, K=9, steps=3)),
    ("fast_bf16_ragged", dict(d=512 * 300 + 8, N=4, n=512, r=4, K=5, steps=3,
                              grad_dtype="bf16", family=1)),
    ("fast_r1", dict(d=64 * 999, N=2, n=64, r=1, K=30, steps=2)),
    ("fast_r2", dict(d=96 * 513, N=5, n=96, r=2, K=7, steps=2)),
    ("fast_r8", dict(d=32 * 4097, N=2, n=32, r=8, K=100, steps=2)),
    ("fast_many_tiles", dict(d=768 * 2600, N=8, n=768, r=4, K=3, steps=2)),
    ("generic_n100_r3", dict(d=100 * 321 + 7, N=3, n=100, r=3, K=12, steps=2)),
    ("generic_odd_d", dict(d=32 * 200 + 3, N=2, n=32, r=4, K=6, steps=2)),
    ("generic_r5_bf16", dict(d=64 * 300, N=2, n=64, r=5, K=4, steps=2, grad_dtype="bf16",
                             family=1)),
    ("n1_exact_like", dict(d=5000, N=3, n=1, r=4, K=50, steps=2)),
    ("k_zero", dict(d=256 * 50, N=2, n=256, r=4, K=0, steps=2)),
    ("k_all", dict(d=256 * 50 + 4, N=2, n=256, r=4, K=51, steps=2)),
    ("k_over", dict(d=256 * 50, N=2, n=256, r=4, K=10_000, steps=2)),
    ("k_one", dict(d=256 * 3000, N=4, n=256, r=4, K=1, steps=2)),
    ("single_worker", dict(d=128 * 640, N=1, n=128, r=4, K=20, steps=2)),
    ("eta_one", dict(d=256 * 80, N=2, n=256, r=4, K=8, eta=1.0, steps=2)),
    ("eta_zero", dict(d=256 * 80, N=2, n=256, r=4, K=8, eta=0.0, steps=2)),
    # one workgroup per bucket up to 32,768 rows, the multi-block radix
    # kernels above that
    ("select_one_workgroup_9000", dict(d=32 * 9000, N=2, n=32, r=4, K=2500, steps=2)),
    ("select_one_workgroup_max", dict(d=8 * 32_768, N=2, n=8, r=4, K=3001, steps=2)),
    ("select_multiblock", dict(d=8 * 32_769, N=2, n=8, r=4, K=3001, steps=2)),
    ("per_worker_N12", dict(d=256 * 300, N=12, n=256, r=4, K=7, steps=2)),
    ("bf16_odd_chunks", dict(d=96 * 700 + 12, N=3, n=96, r=4, K=9, steps=2, grad_dtype="bf16",
                             family=1)),
    ("bf16_per_worker_N9", dict(d=128 * 500, N=9, n=128, r=4, K=6, steps=2, grad_dtype="bf16",
                                family=1)),
    ("bf16_r8_N2", dict(d=64 * 3000, N=2, n=64, r=8, K=40, steps=2, grad_dtype="bf16",
                              family=1)),
    ("select_many_blocks", dict(d=32 * 300_000, N=1, n=32, r=4, K=150_000, steps=1)),
    # worker counts that are multiples of 8 take the one-dimensional
    # (worker, block) grid
    ("flat_grid_N16", dict(d=768 * 400 + 16, N=16, n=768, r=4, K=6, steps=2)),
    ("flat_grid_N24_bf16", dict(d=2048 * 90, N=24, n=2048, r=4, K=4, steps=2,
                                grad_dtype="bf16", family=1)),
    ("generic_r32_max", dict(d=40 * 500 + 13, N=3, n=40, r=32, K=7, steps=2)),
    ("generic_r17_bf16", dict(d=72 * 300 + 5, N=2, n=72, r=17, K=9, steps=2, grad_dtype="bf16",
                              family=1)),
    ("generic_wide_ragged", dict(d=1000 * 70 + 999, N=3, n=1000, r=4, K=5, steps=2)),
    ("generic_many_workers", dict(d=50 * 257, N=11, n=50, r=4, K=20, steps=2)),
    # the sketch kernel with 2 to 6 workers for every r and
    # row-group size (8 rows for n % 256 == 0, 16 for n % 128, 32 for n % 64,
    # 64 otherwise)
    ("r2_g64_N2", dict(d=96 * 513, N=2, n=96, r=2, K=7, steps=2)),
    ("g32_bf16_N3", dict(d=192 * 400, N=3, n=192, r=4, K=9, steps=2, grad_dtype="bf16",
                            family=1)),
    ("per_worker_g32", dict(d=192 * 500, N=4, n=192, r=4, K=9, steps=2)),
    ("per_worker_r8_g64", dict(d=32 * 4097, N=4, n=32, r=8, K=100, steps=2)),
    ("per_worker_r1_bf16", dict(d=128 * 777, N=5, n=128, r=1, K=30, steps=2, grad_dtype="bf16",
                                family=1)),
    ("g8_r8_bf16_N3", dict(d=256 * 700 + 36, N=3, n=256, r=8, K=9, steps=2, grad_dtype="bf16",
                              family=1)),
    ("per_worker_g8_r2", dict(d=512 * 400, N=6, n=512, r=2, K=9, steps=2)),
    ("g16_r4_N2", dict(d=128 * 900, N=2, n=128, r=4, K=9, steps=2)),
    # widths that are multiples of 4 but not of the chunk: every row's last
    # chunk is partial (32 + 4, 64 + 36, 7 x 128 + 104 columns), and the
    # ragged tail row is a one-row vector group as wide as its values
    ("partial_chunk_g64_bf16_N2", dict(d=36 * 900 + 20, N=2, n=36, r=8, K=40, steps=2,
                                          grad_dtype="bf16", family=1)),
    ("partial_chunk_g32_N3", dict(d=100 * 321 + 8, N=3, n=100, r=4, K=12, steps=3)),
    ("partial_chunk_g16_bf16_per_worker", dict(d=1000 * 80 + 996, N=4, n=1000, r=4, K=5, steps=2,
                                               grad_dtype="bf16", family=1)),
    ("partial_chunk_n4_per_worker", dict(d=4 * 5000, N=5, n=4, r=2, K=60, steps=2)),
    ("ragged_tail_r1_per_worker", dict(d=512 * 300 + 12, N=6, n=512, r=1, K=9, steps=2)),
    # rows of 9 or more chunks: workgroups of two waves, one per compute unit
    # (8-, 16-, 32- and 64-row groups, a partial last chunk, a ragged tail row)
    ("two_wave_g8_bf16", dict(d=2304 * 150 + 100, N=3, n=2304, r=4, K=7, steps=2,
                              grad_dtype="bf16", family=1)),
    ("two_wave_g16_bf16_N4", dict(d=2048 * 120, N=4, n=2048, r=4, K=6, steps=2,
                                  grad_dtype="bf16", family=1)),
    ("two_wave_g32_r2", dict(d=576 * 500, N=2, n=576, r=2, K=9, steps=2)),
    ("two_wave_g64_r8", dict(d=288 * 700 + 4, N=2, n=288, r=8, K=12, steps=2)),
    ("two_wave_partial_r1_N5", dict(d=2308 * 100 + 8, N=5, n=2308, r=1, K=4, steps=2)),
    # power-of-two widths in 16-row groups with rows 8 and 2 apart, and a
    # 7-chunk width in 16-row groups of 2 waves with rows 4 apart
    ("pow2_1024_rows8apart", dict(d=1024 * 300 + 4, N=3, n=1024, r=4, K=5, steps=2)),
    ("pow2_4096_rows2apart_bf16", dict(d=4096 * 80, N=2, n=4096, r=4, K=3, steps=2,
                                        grad_dtype="bf16", family=1)),
    ("g16_896_two_wave_r2", dict(d=896 * 150, N=3, n=896, r=2, K=6, steps=2)),
    # the widest rows the vectorised kernels take (2^22 values, plus a ragged
    # tail row of half that), and 4 values more, which go to the general one
    ("max_width_vector", dict(d=(1 << 22) * 3 + (1 << 21), N=2, n=1 << 22, r=4, K=2, steps=2)),
    ("over_max_width_general", dict(d=((1 << 22) + 4) * 2, N=2, n=(1 << 22) + 4, r=4, K=1,
                                    steps=1)),
]


@pytest.mark.parametrize("name,kw", CASES, ids=[c[0] for c in CASES])
def test_parity_small(name, kw):
    log(f"[parity] {name} {kw}")
    run_case(label=name, check_S=True, **kw)


def test_describe_names_the_kernel_path():
    for N, want in ((1, "sketch=per_worker+reduce"), (3, "sketch=per_worker+reduce"),
                    (4, "sketch=per_worker+reduce"),
                    (8, "sketch=per_worker+reduce"), (12, "sketch=per_worker+reduce")):
        comp = arc.Compressor(d=256 * 64, N=N, n=256, K=3, eta=0.1, seed=1)
        try:
            desc = comp.describe()
            log(f"[describe] N={N}: {desc}")
            assert want in desc, desc
        finally:
            comp.close()
    comp = arc.Compressor(d=100 * 64, N=2, n=100, r=3, K=3, eta=0.1, seed=1)
    try:
        assert "sketch=general" in comp.describe()
    finally:
        comp.close()
    # one workgroup per bucket up to 32,768 rows, then the multi-block kernels
    for rows, want in ((32_768, "select=one_workgroup_per_bucket"), (32_769, "select=blocks:5")):
        comp = arc.Compressor(d=8 * rows, N=1, n=8, K=3, eta=0.1, seed=1)
        try:
            assert want in comp.describe(), comp.describe()
        finally:
            comp.close()
    # the widest vectorised rows, and one step wider
    for n, want in ((1 << 22, "general_groups=0"), ((1 << 22) + 4, "sketch=general")):
        comp = arc.Compressor(d=n * 2, N=2, n=n, r=4, K=1, eta=0.1, seed=1)
        try:
            assert want in comp.describe(), comp.describe()
        finally:
            comp.close()
    # launch shapes: one 256-column chunk per row runs uncapped, 3 chunks in
    # 4-wave workgroups and 16 chunks in 2-wave ones, one per compute unit
    # and 16-chunk rows in groups of every 4th row of a block of 4 groups;
    # power-of-two widths from 1024 take 16-row groups whose rows lie 32 KiB
    # apart (8 rows apart at 1024 values)
    for n, rows, want, strided in ((256, 70, "workgroup_waves=(4 4 4 4)", 0),
                                   (768, 70, "workgroup_waves=(4 4 4 4/cu)", 0),
                                   (2048, 70, "workgroup_waves=(4 4 2/cu 4)", 4),
                                   (1024, 140, "workgroup_waves=(4 4 2/cu 4)", 8)):
        comp = arc.Compressor(d=n * rows, N=2, n=n, r=4, K=3, eta=0.1, seed=1)
        try:
            desc = comp.describe()
            assert want in desc, desc
            assert f"interleaved_groups={strided} " in desc, desc
        finally:
            comp.close()
    # a width that is a multiple of 4 but of no chunk width, with a ragged
    # tail row: all vector groups, no general kernel
    comp = arc.Compressor(d=100 * 64 + 8, N=2, n=100, r=4, K=3, eta=0.1, seed=1)
    try:
        desc = comp.describe()
        assert "sketch=per_worker+reduce" in desc and "general_groups=0" in desc, desc
    finally:
        comp.close()


def test_parity_steps_out_of_order():
    # The library generates step t+1's projection while step t runs; a caller
    # that skips, repeats or goes back in t gets V_t generated on the spot.
    ts = [0, 1, 2, 7, 8, 3, 3, 0, 1]
    run_case(label="out_of_order_single", d=256 * 300 + 40, N=3, n=256, r=4, K=9, ts=ts)
    run_case(label="out_of_order_tensors", d=sum(a * b for a, b, _ in TENSORS_3W), N=4, r=4,
             tensors=TENSORS_3W, ts=ts)


TENSORS_3W = [(300, 64, 5), (40, 1000, 3), (129, 256, 4), (1, 2048, 1)]


@pytest.mark.parametrize("n,rows", [(256, 120), (2304, 70)])
def test_parity_misaligned_pointers_take_the_general_path(n, rows):
    # 2304-wide rows: the vectorised plan's groups take every 4th row of a
    # block of 32, and the general kernel must follow them
    log(f"[parity] misaligned n={n}")
    run_case(label=f"misaligned_{n}", d=n * rows, N=3, n=n, r=4, K=11, steps=2, misalign=1)


# Pointers 16-byte aligned but 16 to 112 bytes past a 128-byte line, and
# worker bases further off the lines (d = rows * n + 40): the 8- and 16-row
# groups shift their column windows onto whole lines, a row's first and last
# windows partial.
@pytest.mark.parametrize("n,rows,dtype,mis", [
    (512, 300, "f32", 4), (512, 300, "f32", 28), (768, 200, "f32", 12),
    (256, 400, "bf16", 8), (2048, 80, "bf16", 24), (4096, 40, "f32", 16),
    (1536, 90, "bf16", 16)])
def test_parity_line_shifted_windows(n, rows, dtype, mis):
    log(f"[parity] shifted windows n={n} {dtype} misalign={mis}")
    run_case(label=f"shifted_{n}_{dtype}_{mis}", d=n * rows + 40, N=3, n=n, r=4, K=13,
             steps=2, grad_dtype=dtype, family=1 if dtype == "bf16" else 0, misalign=mis,
             check_S=True)


def test_parity_buckets():
    # buckets: radix, dense (K >= rows), empty selection, one-row bucket
    n = 64
    begin = [0, 1000, 1300, 1301, 5000, 6000]
    ks = [17, 500, 1, 0, 10]
    d = n * 6000
    log("[parity] buckets")
    run_case(label="buckets", d=d, N=3, n=n, r=4, buckets=(begin, ks), steps=3)


# Selections over at most 32,768 rows per bucket take the one-workgroup path,
# larger ones the multi-block radix kernels: both sizes for the tie cases.
@pytest.mark.parametrize("rows", [400, 20_000, 40_000])
def test_parity_zero_residual_ties_take_lowest_rows(rows):
    d, N, n = 32 * rows, 2, 32
    zero = np.zeros((N, d), F32)
    log(f"[parity] zero residual, {rows} rows")
    run_case(label=f"zeros_{rows}", d=d, N=N, n=n, K=13, steps=2, grad_fn=lambda t: zero)


@pytest.mark.parametrize("rows,K", [(5000, 1234), (32_768, 9_001), (70_000, 17_321)])
def test_parity_crafted_ties(rows, K):
    # V = ones (r = 1): Sigma_p = (sum over workers and row of Delta)^2, built
    # from small integers so that many rows tie exactly at the threshold.
    d, N, n = 32 * rows, 2, 32
    rng = np.random.default_rng(5)
    vals = rng.integers(0, 4, size=(rows,)).astype(F32)  # row sums in {0..3}

    def grad(t):
        g = np.zeros((N, d), F32)
        g[0, ::n] = vals  # first column of each row for worker 0
        return g

    log(f"[parity] crafted ties, {rows} rows")
    run_case(label=f"ties_{rows}", d=d, N=N, n=n, r=1, K=K, eta=1.0, steps=1, grad_fn=grad,
             V=np.ones((n, 1), F32))


# A bucket of more than 256 blocks x 8192 rows (2,097,152) gives every
# selection block more than one tile of keys (here 9,984 rows a block: a
# full tile and a partial one); the ties at the threshold then run across
# tiles as well as blocks.
@pytest.mark.parametrize("kind", ["zeros", "ties"])
def test_parity_multi_tile_selection_blocks(kind):
    rows, n, N = 2_500_000, 4, 2
    d = n * rows
    log(f"[parity] multi-tile selection blocks, {kind}")
    if kind == "zeros":
        zero = np.zeros((N, d), F32)
        run_case(label="zeros_multitile", d=d, N=N, n=n, K=2_400_001, steps=2,
                 grad_fn=lambda t: zero)
        return
    rng = np.random.default_rng(6)
    vals = rng.integers(0, 4, size=(rows,)).astype(F32)

    def grad(t):
        g = np.zeros((N, d), F32)
        g[0, ::n] = vals
        return g

    run_case(label="ties_multitile", d=d, N=N, n=n, r=1, K=1_000_003, eta=1.0, steps=1,
             grad_fn=grad, V=np.ones((n, 1), F32))


def test_parity_injected_projection():
    rng = np.random.default_rng(9)
    V = rng.standard_normal((256, 4)).astype(F32)
    log("[parity] injected V")
    run_case(label="injected_V", d=256 * 333, N=3, n=256, K=10, steps=2, V=V)


def test_library_projection_matches_oracle_bitwise():
    comp = arc.Compressor(d=768 * 10, N=1, n=768, r=4, K=1, eta=0.1, seed=2003)
    try:
        for t in (0, 1, 19, 123456):
            got = np.empty((768, 4), F32)
            arc.arc_debug_projection(comp.ctx, t, got)
            want = oracle.projection(2003, t, 768, 4)
            assert got.tobytes() == want.tobytes(), t
    finally:
        comp.close()


def test_repeat_is_bit_identical():
    # Same inputs twice: every output identical (no scheduling dependence).
    d, N, n, K = 512 * 2000, 4, 512, 40
    gen = synth.Generator(d, N, 3)
    grad = torch.from_numpy(gen.fill_host(0)).cuda()
    outs = []
    for _ in range(2):
        comp = arc.Compressor(d=d, N=N, n=n, K=K, eta=0.1, seed=5)
        h = torch.zeros((N, d), device="cuda")
        g = torch.zeros((N, d), device="cuda")
        idx, agg = comp.step(0, grad, h, g)
        sig = comp.sigma()
        torch.cuda.synchronize()
        outs.append([x.cpu().numpy().tobytes() for x in (idx, agg, sig, h, g)])
        comp.close()
    assert outs[0] == outs[1]


def test_step_rejects_overlapping_buffers():
    d, N = 256 * 10, 2
    comp = arc.Compressor(d=d, N=N, n=256, K=2, eta=0.1, seed=5)
    try:
        h = torch.zeros((N, d), device="cuda")
        g = torch.zeros((N, d), device="cuda")
        with pytest.raises(arc.ArcError, match="overlap"):
            arc.arc_step(comp.ctx, 0, h, h, g, comp.idx, comp.agg)
        with pytest.raises(arc.ArcError, match="overlap"):
            arc.arc_step(comp.ctx, 0, g, h, g, comp.idx, comp.agg)
        with pytest.raises(arc.ArcError, match="t must be"):
            arc.arc_step(comp.ctx, -1, torch.zeros_like(h), h, g, comp.idx, comp.agg)
        # outputs aliasing each other or the state: rejected before any work
        grad = torch.ones((N, d), device="cuda")
        h0, g0 = h.clone(), g.clone()
        for idx, agg in ((h, comp.agg), (comp.idx, g), (grad, comp.agg), (comp.idx, grad),
                         (comp.idx, comp.idx), (comp.agg[1:], comp.agg)):
            with pytest.raises(arc.ArcError, match="overlap"):
                arc.arc_step(comp.ctx, 0, grad, h, g, idx, agg)
        torch.cuda.synchronize()
        assert torch.equal(h, h0) and torch.equal(g, g0)
    finally:
        comp.close()


def test_device_generator_matches_host_generator():
    for kw in (dict(d=1 << 20, N=3, seed=1001, per_coord_scale=True, noise=0.3),
               dict(d=11_689_512 // 8, N=2, seed=1002, noise=0.5, scale_sigma=1.5,
                    boost=20.0, boost_frac=0.001),
               dict(d=2048 * 300, N=4, seed=1004, grad_dtype="bf16", family=1,
                    tensors=[2048 * 100, 2048 * 150, 2048 * 50])):
        gen = synth.Generator(**kw)
        for t in (0, 3):
            dt = torch.int16 if gen.grad_dtype == "bf16" else torch.float32
            out = torch.empty((gen.N, gen.d), dtype=dt, device="cuda")
            gen.fill_device(t, out)
            torch.cuda.synchronize()
            dev_np = out.cpu().numpy().view(gen.np_dtype)
            host_np = gen.fill_host(t)
            assert dev_np.tobytes() == host_np.tobytes(), (kw, t)


def test_two_contexts_on_two_streams_interleaved():
    # Two compressors, each bound to its own stream (with its own side stream
    # and projection staging), stepped alternately with no synchronisation in
    # between: each must still match its own oracle run.
    from parity_util import compare_float, to_device_grad

    dev = torch.device("cuda:0")
    cfgs = [dict(d=2304 * 70 + 100, N=3, n=2304, K=5, grad_dtype="bf16", family=1,
                 data_seed=31, seed=5),
            dict(d=768 * 300, N=2, n=768, K=7, grad_dtype="f32", family=0, data_seed=32,
                 seed=6)]
    steps = 3
    streams = [torch.cuda.Stream(dev) for _ in cfgs]
    comps, hs, gs, grads = [], [], [], []
    try:
        for c, s in zip(cfgs, streams):
            comps.append(arc.Compressor(d=c["d"], N=c["N"], n=c["n"], r=4, K=c["K"], eta=0.1,
                                        seed=c["seed"], grad_dtype=c["grad_dtype"], device=dev,
                                        stream=s))
            gen = synth.Generator(c["d"], c["N"], c["data_seed"], grad_dtype=c["grad_dtype"],
                                  family=c["family"])
            grads.append([gen.fill_host(t) for t in range(steps)])
            hs.append(torch.zeros((c["N"], c["d"]), device=dev))
            gs.append(torch.zeros((c["N"], c["d"]), device=dev))
        dgrads = [[to_device_grad(x, dev) for x in gr] for gr in grads]
        torch.cuda.synchronize(dev)
        outs = [[], []]
        for t in range(steps):
            for k in range(2):
                with torch.cuda.stream(streams[k]):
                    idx, agg = comps[k].step(t, dgrads[k][t], hs[k], gs[k])
                    outs[k].append((idx.clone(), agg.clone()))
        torch.cuda.synchronize(dev)
        for k, c in enumerate(cfgs):
            log(f"[parity] two streams: context {k} {c}")
            h_o = np.zeros((c["N"], c["d"]), F32)
            g_o = np.zeros((c["N"], c["d"]), F32)
            for t in range(steps):
                want = oracle.step(h_o, g_o, grads[k][t], n=c["n"], r=4, eta=0.1, seed=c["seed"],
                                   t=t, K=c["K"])
                assert np.array_equal(outs[k][t][0].cpu().numpy(), want["idx"]), (k, t)
                compare_float(f"ctx{k} t={t} agg", outs[k][t][1].cpu().numpy(), want["agg"])
            compare_float(f"ctx{k} h", hs[k].cpu().numpy(), h_o)
            compare_float(f"ctx{k} g", gs[k].cpu().numpy(), g_o)
    finally:
        for comp in comps:
            comp.close()


@pytest.mark.parametrize("tensors", [False, True], ids=["single_view", "tensors"])
def test_steps_queued_ahead_of_a_busy_device(tensors):
    # The host queues many steps while the device is still busy with earlier
    # work, so every staging buffer of the projection ring is refilled while
    # earlier steps are in flight (and, out of order, generated on the spot):
    # every step must still use its own V_t.
    from parity_util import compare_float, to_device_grad

    dev = torch.device("cuda:0")
    stream = torch.cuda.Stream(dev)
    if tensors:
        kw = dict(d=sum(a * b for a, b, _ in TENSORS_3W), N=3, tensors=TENSORS_3W)
    else:
        kw = dict(d=512 * 400 + 8, N=3, n=512, K=9)
    ts = [0, 1, 2, 3, 4, 5, 9, 10, 11, 12, 4, 13, 14]
    gen = synth.Generator(kw["d"], kw["N"], 41,
                          tensors=None if not tensors else [a * b for a, b, _ in TENSORS_3W])
    grads = [gen.fill_host(t) for t in range(len(ts))]
    comp = arc.Compressor(r=4, eta=0.1, seed=12, device=dev, stream=stream, **kw)
    try:
        dgrads = [to_device_grad(x, dev) for x in grads]
        h = torch.zeros((kw["N"], kw["d"]), device=dev)
        g = torch.zeros((kw["N"], kw["d"]), device=dev)
        big = torch.randn(4096, 4096, device=dev)
        torch.cuda.synchronize(dev)
        outs = []
        with torch.cuda.stream(stream):
            for _ in range(8):  # keep the device busy while the host queues the steps
                big = big @ big * (1.0 / 64.0)
            for k, t in enumerate(ts):
                idx, agg = comp.step(t, dgrads[k], h, g)
                outs.append((idx.clone(), agg.clone()))
        torch.cuda.synchronize(dev)
        h_o = np.zeros((kw["N"], kw["d"]), F32)
        g_o = np.zeros((kw["N"], kw["d"]), F32)
        for k, t in enumerate(ts):
            if tensors:
                want = oracle.step_tensors(h_o, g_o, grads[k], TENSORS_3W, r=4, eta=0.1, seed=12,
                                           t=t)
            else:
                want = oracle.step(h_o, g_o, grads[k], n=kw["n"], r=4, eta=0.1, seed=12, t=t,
                                   K=kw["K"])
            assert np.array_equal(outs[k][0].cpu().numpy(), want["idx"]), (k, t)
            compare_float(f"queued t={t} agg", outs[k][1].cpu().numpy(), want["agg"])
        compare_float("queued h", h.cpu().numpy(), h_o)
        compare_float("queued g", g.cpu().numpy(), g_o)
    finally:
        comp.close()
