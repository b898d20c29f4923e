"""ctypes binding of libarctopk (include/libarctopk.h): argument marshalling only.

Every stage of the compressor runs in the HIP library.  Importing this module
fails loudly when ``libarctopk.so`` has not been built; there is no fallback.
Device buffers may be passed as torch tensors (their ``data_ptr()`` is used) or
as integer device addresses.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libarctopk.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(
        f"{LIB_PATH} is missing: build the HIP library first "
        "(python -c 'import __graft_entry__ as g; g.build()')")

# One HIP runtime per process: torch ships its own libamdhip64, and a second
# copy loaded beside it makes both fail.  Loading torch first makes
# libarctopk resolve to the runtime torch already holds, so the two share
# devices and streams.  Without torch the system runtime is used.
try:
    import torch  # noqa: F401
except ImportError:  # pragma: no cover - torch-free use of the C library
    pass

_lib = ctypes.CDLL(LIB_PATH)

ARC_OK, ARC_ERR_INVALID, ARC_ERR_NOMEM, ARC_ERR_DEVICE, ARC_ERR_UNSUPPORTED = 0, 1, 2, 3, 4
ARC_DTYPE_F32, ARC_DTYPE_BF16 = 0, 1
ARC_MAX_R = 32
ARC_STATIC_SCRATCH_BYTES = 64 * 1024 * 1024
ARC_NUM_STAGES = 5
STAGE_NAMES = ("sketch", "reduce", "select", "gather_update", "step")


class arc_tensor(ctypes.Structure):
    _fields_ = [
        ("rows", ctypes.c_int64),
        ("cols", ctypes.c_int64),
        ("K", ctypes.c_int64),
    ]


class arc_config(ctypes.Structure):
    _fields_ = [
        ("d", ctypes.c_int64),
        ("n", ctypes.c_int64),
        ("K", ctypes.c_int64),
        ("seed", ctypes.c_uint64),
        ("bucket_row_begin", ctypes.POINTER(ctypes.c_int64)),
        ("bucket_K", ctypes.POINTER(ctypes.c_int64)),
        ("N", ctypes.c_int32),
        ("r", ctypes.c_int32),
        ("grad_dtype", ctypes.c_int32),
        ("num_buckets", ctypes.c_int32),
        ("eta", ctypes.c_float),
        ("reserved", ctypes.c_int32),
        ("tensors", ctypes.POINTER(arc_tensor)),
        ("num_tensors", ctypes.c_int32),
        ("compressor", ctypes.c_int32),
    ]


ARC_COMP_ARC, ARC_COMP_RANDK, ARC_COMP_TOPK = 0, 1, 2
COMPRESSORS = {"arc": ARC_COMP_ARC, "randk": ARC_COMP_RANDK, "topk": ARC_COMP_TOPK}
ARC_OPT_SGD, ARC_OPT_MSGD, ARC_OPT_ADAM = 0, 1, 2
OPTIMIZERS = {"sgd": ARC_OPT_SGD, "msgd": ARC_OPT_MSGD, "adam": ARC_OPT_ADAM}


class arc_model_config(ctypes.Structure):
    _fields_ = [
        ("optimizer", ctypes.c_int32),
        ("dense_steps", ctypes.c_int32),
        ("lr", ctypes.c_float),
        ("momentum", ctypes.c_float),
        ("beta1", ctypes.c_float),
        ("beta2", ctypes.c_float),
        ("eps", ctypes.c_float),
        ("weight_decay", ctypes.c_float),
    ]


def make_model_config(optimizer="sgd", *, lr, dense_steps=0, momentum=0.0, beta1=0.9,
                      beta2=0.999, eps=1e-8, weight_decay=0.0) -> arc_model_config:
    kind = OPTIMIZERS[optimizer] if isinstance(optimizer, str) else int(optimizer)
    return arc_model_config(kind, dense_steps, lr, momentum, beta1, beta2, eps, weight_decay)


_st = ctypes.c_int
_vp = ctypes.c_void_p
_SIGS = {
    "arc_create": (_st, [ctypes.POINTER(arc_config), _vp, ctypes.POINTER(_vp)]),
    "arc_step": (_st, [_vp, ctypes.c_int64, _vp, _vp, _vp, _vp, _vp]),
    "arc_model_step": (_st, [_vp, ctypes.POINTER(arc_model_config), ctypes.c_int64, _vp, _vp,
                             _vp, _vp, _vp, _vp, _vp, _vp, _vp]),
    "arc_step_static": (_st, [ctypes.POINTER(arc_config), _vp, ctypes.c_int64, _vp, _vp, _vp,
                              _vp, _vp]),
    "arc_destroy": (_st, [_vp]),
    "arc_num_rows": (ctypes.c_int64, [_vp]),
    "arc_selected_rows": (ctypes.c_int64, [_vp]),
    "arc_payload_elems": (ctypes.c_int64, [_vp]),
    "arc_projection": (_st, [ctypes.c_uint64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                             _vp]),
    "arc_status_str": (ctypes.c_char_p, [_st]),
    "arc_last_error": (ctypes.c_char_p, []),
    "arc_describe": (_st, [_vp, ctypes.c_char_p, ctypes.c_int64]),
    "arc_debug_sigma": (_st, [_vp, _vp]),
    "arc_debug_sketch": (_st, [_vp, _vp]),
    "arc_debug_projection": (_st, [_vp, ctypes.c_int64, _vp]),
    "arc_set_projection": (_st, [_vp, _vp]),
    "arc_timing_enable": (_st, [_vp, ctypes.c_int32]),
    "arc_timing_read": (_st, [_vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)]),
}
for _name, (_res, _args) in _SIGS.items():
    _fn = getattr(_lib, _name)
    _fn.restype = _res
    _fn.argtypes = _args

EXPORTED = tuple(_SIGS)


class ArcError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        name = _lib.arc_status_str(status).decode()
        detail = _lib.arc_last_error().decode()
        super().__init__(f"{where}: {name}: {detail}")


def _check(status: int, where: str) -> None:
    if status != ARC_OK:
        raise ArcError(status, where)


def _addr(x):
    """Device/host address of a tensor, numpy array or integer (None -> NULL)."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    if hasattr(x, "ctypes"):
        return x.ctypes.data
    raise TypeError(f"cannot take the address of {type(x)!r}")


def make_config(*, d: int, N: int, n: int = 0, r: int = 4, K: int = 0, eta: float,
                seed: int, grad_dtype: int = ARC_DTYPE_F32, buckets=None, tensors=None,
                reserved: int = 0, compressor=0):
    """Build an ``arc_config``; ``buckets`` = (row_begin[nb+1], K[nb]) or None;
    ``tensors`` = [(rows, cols, K), ...] for the per-tensor mode (then n, K
    and buckets stay 0 / None); ``compressor`` = "arc", "randk" or "topk".  Returns (config, keepalive) - keep the second
    value alive until arc_create returns (it owns the arrays)."""
    cfg = arc_config(d=d, n=n, K=K, seed=seed & (2**64 - 1), N=N, r=r,
                     grad_dtype=grad_dtype, num_buckets=0, eta=eta, reserved=reserved,
                     num_tensors=0, compressor=COMPRESSORS.get(compressor, compressor))
    keep = []
    if buckets is not None:
        begin, ks = buckets
        b_arr = (ctypes.c_int64 * len(begin))(*begin)
        k_arr = (ctypes.c_int64 * len(ks))(*ks)
        cfg.bucket_row_begin = ctypes.cast(b_arr, ctypes.POINTER(ctypes.c_int64))
        cfg.bucket_K = ctypes.cast(k_arr, ctypes.POINTER(ctypes.c_int64))
        cfg.num_buckets = len(ks)
        keep += [b_arr, k_arr]
    if tensors is not None:
        t_arr = (arc_tensor * len(tensors))(*[arc_tensor(int(a), int(b), int(c))
                                             for a, b, c in tensors])
        cfg.tensors = ctypes.cast(t_arr, ctypes.POINTER(arc_tensor))
        cfg.num_tensors = len(tensors)
        keep.append(t_arr)
    return cfg, keep


def arc_create(cfg: arc_config, hip_stream=None) -> int:
    """Returns the context handle (an integer).  ``hip_stream``: a torch stream,
    a raw hipStream_t integer, or None for the default stream."""
    stream = getattr(hip_stream, "cuda_stream", hip_stream)
    out = _vp()
    _check(_lib.arc_create(ctypes.byref(cfg), stream, ctypes.byref(out)), "arc_create")
    return out.value


def arc_step(ctx: int, t: int, grad, h, g, out_idx, out_agg) -> None:
    _check(_lib.arc_step(ctx, t, _addr(grad), _addr(h), _addr(g), _addr(out_idx),
                         _addr(out_agg)), "arc_step")


def arc_step_static(cfg: arc_config, stream, t: int, grad, h, g, out_idx, out_agg) -> None:
    """The allocation-free step: no context, device scratch in the library's
    static array.  stream: a torch stream, a raw hipStream_t or None."""
    _check(_lib.arc_step_static(ctypes.byref(cfg), getattr(stream, "cuda_stream", stream), t,
                                _addr(grad),
                                _addr(h), _addr(g), _addr(out_idx), _addr(out_agg)),
           "arc_step_static")


def arc_model_step(ctx: int, mc: arc_model_config, t: int, grad, h, g, G, x, opt_m, opt_v,
                   out_idx, out_agg) -> None:
    _check(_lib.arc_model_step(ctx, ctypes.byref(mc), t, _addr(grad), _addr(h), _addr(g),
                               _addr(G), _addr(x), _addr(opt_m), _addr(opt_v), _addr(out_idx),
                               _addr(out_agg)), "arc_model_step")


def arc_destroy(ctx) -> None:
    _check(_lib.arc_destroy(ctx), "arc_destroy")


def arc_num_rows(ctx) -> int:
    return int(_lib.arc_num_rows(ctx))


def arc_selected_rows(ctx) -> int:
    return int(_lib.arc_selected_rows(ctx))


def arc_payload_elems(ctx) -> int:
    return int(_lib.arc_payload_elems(ctx))


def arc_projection(seed: int, t: int, n: int, r: int, out_V) -> None:
    """V_t of width n for a shared seed into host memory (numpy [n, r] f32)."""
    _check(_lib.arc_projection(seed & (2**64 - 1), t, n, r, _addr(out_V)), "arc_projection")


def arc_status_str(status: int) -> str:
    return _lib.arc_status_str(status).decode()


def arc_last_error() -> str:
    return _lib.arc_last_error().decode()


def arc_describe(ctx) -> str:
    buf = ctypes.create_string_buffer(512)
    _check(_lib.arc_describe(ctx, buf, len(buf)), "arc_describe")
    return buf.value.decode()


def arc_debug_sigma(ctx, out_sigma) -> None:
    _check(_lib.arc_debug_sigma(ctx, _addr(out_sigma)), "arc_debug_sigma")


def arc_debug_sketch(ctx, out_S) -> None:
    _check(_lib.arc_debug_sketch(ctx, _addr(out_S)), "arc_debug_sketch")


def arc_debug_projection(ctx, t: int, out_V) -> None:
    _check(_lib.arc_debug_projection(ctx, t, _addr(out_V)), "arc_debug_projection")


def arc_set_projection(ctx, V) -> None:
    _check(_lib.arc_set_projection(ctx, _addr(V)), "arc_set_projection")


def arc_timing_enable(ctx, on: bool) -> None:
    _check(_lib.arc_timing_enable(ctx, 1 if on else 0), "arc_timing_enable")


def arc_timing_read(ctx):
    """Returns (ms_per_stage_sum[5], steps)."""
    ms = (ctypes.c_double * ARC_NUM_STAGES)()
    steps = ctypes.c_int64(0)
    _check(_lib.arc_timing_read(ctx, ms, ctypes.byref(steps)), "arc_timing_read")
    return list(ms), steps.value


def raw_status(name: str, *args) -> int:
    """Call an entry point and return its raw status (for error-path tests)."""
    return int(getattr(_lib, name)(*args))
