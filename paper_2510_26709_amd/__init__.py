"""libarctopk: the ARC-Top-K + EF21M compressor step (arXiv:2510.26709) as
hand-written HIP kernels for the AMD Instinct MI355X (gfx950).

The library is the C ABI declared in ``include/libarctopk.h``; this package is
its ctypes binding (same entry-point names) plus ``Compressor``, a small owner
of a context and its output buffers.  All compute runs in ``libarctopk.so``.
"""
from __future__ import annotations

from ._lib import (  # noqa: F401
    ARC_DTYPE_BF16, ARC_DTYPE_F32, ARC_ERR_DEVICE, ARC_ERR_INVALID, ARC_ERR_NOMEM,
    ARC_COMP_ARC, ARC_COMP_RANDK, ARC_COMP_TOPK, ARC_ERR_UNSUPPORTED, ARC_MAX_R, COMPRESSORS, ARC_NUM_STAGES, ARC_OK, ARC_OPT_ADAM, ARC_OPT_MSGD,
    ARC_OPT_SGD, EXPORTED, LIB_PATH, OPTIMIZERS, STAGE_NAMES, ArcError, arc_config, arc_create,
    arc_debug_projection, arc_describe, arc_debug_sigma, arc_debug_sketch, arc_destroy,
    arc_last_error, arc_model_config, arc_model_step, arc_num_rows, arc_payload_elems,
    arc_projection, arc_selected_rows, arc_set_projection, arc_status_str, arc_step,
    arc_step_static, ARC_STATIC_SCRATCH_BYTES, arc_tensor,
    arc_timing_enable, arc_timing_read, make_config, make_model_config)


class Compressor:
    """One libarctopk context bound to a torch stream, with its outputs.

    ``step(t, grad, h, g)`` enqueues one compressor step and returns the
    device tensors idx [K_total] int32 and agg, overwritten by the next step:
    [K_total, n] float32 for one m x n view, or, with ``tensors`` =
    [(rows, cols, K), ...] (per-tensor mode), the packed 1-D payload.  With
    ``compressor="topk"`` both gain a leading node axis: idx [N, K] and agg
    [N, K, n] (or [N, L] packed).
    """

    def __init__(self, *, d, N, n=0, r=4, K=0, eta, seed, grad_dtype="f32", buckets=None,
                 tensors=None, compressor="arc", device=None, stream=None):
        import torch
        self.device = torch.device(device or "cuda")
        self.stream = stream or torch.cuda.current_stream(self.device)
        dt = ARC_DTYPE_BF16 if grad_dtype == "bf16" else ARC_DTYPE_F32
        cfg, keep = make_config(d=d, N=N, n=n, r=r, K=K, eta=eta, seed=seed, grad_dtype=dt,
                                buckets=buckets, tensors=tensors, compressor=compressor)
        self.compressor = compressor
        with torch.cuda.device(self.device):
            self.ctx = arc_create(cfg, self.stream)
        del keep
        self.d, self.N, self.n, self.r = d, N, n, r
        self.tensors = None if tensors is None else [tuple(map(int, x)) for x in tensors]
        self.m = arc_num_rows(self.ctx)
        self.K_total = arc_selected_rows(self.ctx)
        self.payload = arc_payload_elems(self.ctx)
        self.idx = torch.empty(max(self.K_total, 1), dtype=torch.int32, device=self.device)
        self.agg = torch.empty(max(self.payload, 1), dtype=torch.float32, device=self.device)

    def _outputs(self):
        idx, agg = self.idx[: self.K_total], self.agg[: self.payload]
        if self.compressor == "topk":  # one list of rows and values per node
            idx = idx.view(self.N, self.K_total // self.N)
            agg = agg.view(self.N, self.payload // self.N)
            if self.tensors is None:
                agg = agg.view(self.N, self.K_total // self.N, self.n)
        elif self.tensors is None:
            agg = agg.view(self.K_total, self.n)
        return idx, agg

    def step(self, t, grad, h, g):
        arc_step(self.ctx, t, grad, h, g, self.idx, self.agg)
        return self._outputs()

    def model_step(self, t, grad, h, g, G, x, mc, opt_m=None, opt_v=None):
        """One EF21M iteration with the model update (arc_model_step); mc is an
        arc_model_config (see make_model_config).  Returns (idx, agg) as step()
        does; on dense iterations they are not written."""
        arc_model_step(self.ctx, mc, t, grad, h, g, G, x, opt_m, opt_v, self.idx, self.agg)
        return self._outputs()

    def describe(self):
        return arc_describe(self.ctx)

    def sigma(self):
        import torch
        out = torch.empty(self.m, dtype=torch.float32, device=self.device)
        arc_debug_sigma(self.ctx, out)
        return out

    def sketch(self):
        import torch
        out = torch.empty((self.N, self.m, self.r), dtype=torch.float32, device=self.device)
        arc_debug_sketch(self.ctx, out)
        return out

    def close(self):
        if getattr(self, "ctx", None):
            arc_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
