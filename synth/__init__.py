"""Seeded synthetic gradients for the compressor's tests and benchmark.

Input generation only: this package holds none of the compressor's arithmetic.
It serves both sides of the parity tests (the oracle's inputs and the GPU
library's inputs).  The host fill (C, OpenMP) and the device fill (HIP) run
the same exact-operation recipe (``synth_core.h``) and produce identical bits;
a GPU test checks that.

Recipes (per workload; t = step, i = worker, j = coordinate):
  family 0:  g_i[j] = b_j * s(j) * (m_j + noise * e_ij),  m, e ~ N(0,1) fresh per step
  family 1:  g_i[j] = s(j) * (sqrt(c) T_j + sqrt(1-c) T_ij),  T ~ Student-t(3)
with s(j) ~ LogNormal(0, sigma) drawn once per run (per coordinate or per
tensor) and b_j the optional boost of a seeded fraction of coordinates.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from .workloads import ORDER, WORKLOADS, Workload  # noqa: F401

_HERE = os.path.dirname(os.path.abspath(__file__))
_HOST_LIB = os.path.join(_HERE, "libsynth_host.so")
_DEV_LIB = os.path.join(_HERE, "libsynth_dev.so")
_host = None
_dev = None

STREAM_SCALE_COORD = 10
STREAM_SCALE_TENSOR = 11


class _Plan(ctypes.Structure):
    _fields_ = [("family", ctypes.c_int32), ("out_bf16", ctypes.c_int32),
                ("d", ctypes.c_int64), ("N", ctypes.c_int32), ("per_coord", ctypes.c_int32),
                ("seed", ctypes.c_uint64), ("noise", ctypes.c_float),
                ("c_shared", ctypes.c_float), ("c_own", ctypes.c_float),
                ("boost", ctypes.c_float), ("boost_threshold", ctypes.c_uint32),
                ("nseg", ctypes.c_int32), ("seg_begin", ctypes.c_void_p),
                ("scale", ctypes.c_void_p)]


def _host_lib():
    global _host
    if _host is None:
        if not os.path.exists(_HOST_LIB):
            raise ImportError(f"{_HOST_LIB} missing: run __graft_entry__.build()")
        lib = ctypes.CDLL(_HOST_LIB)
        lib.synth_fill_host.restype = ctypes.c_int
        lib.synth_fill_host.argtypes = [ctypes.POINTER(_Plan), ctypes.c_int64, ctypes.c_int32,
                                        ctypes.c_int32, ctypes.c_int64, ctypes.c_int64,
                                        ctypes.c_void_p, ctypes.c_int64]
        lib.synth_normals_host.restype = ctypes.c_int
        lib.synth_normals_host.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int64,
                                           ctypes.c_void_p]
        _host = lib
    return _host


def _dev_lib():
    global _dev
    if _dev is None:
        import torch  # noqa: F401  (share torch's HIP runtime; see paper_2510_26709_amd._lib)
        if not os.path.exists(_DEV_LIB):
            raise ImportError(f"{_DEV_LIB} missing: run __graft_entry__.build()")
        lib = ctypes.CDLL(_DEV_LIB)
        lib.synth_fill_device.restype = ctypes.c_int
        lib.synth_fill_device.argtypes = [ctypes.POINTER(_Plan), ctypes.c_int64,
                                          ctypes.c_void_p, ctypes.c_void_p]
        _dev = lib
    return _dev


def normals(seed: int, stream: int, n: int) -> np.ndarray:
    out = np.empty(n, dtype=np.float32)
    if _host_lib().synth_normals_host(seed, stream, n, out.ctypes.data) != 0:
        raise ValueError("synth_normals_host failed")
    return out


class Generator:
    """Gradient generator for one workload shape.

    ``tensors``: per-tensor sizes (segments with their own scale); ``None`` with
    ``per_coord_scale`` gives one scale per coordinate; ``None`` otherwise gives
    a single segment.
    """

    def __init__(self, d: int, N: int, seed: int, *, grad_dtype: str = "f32", family: int = 0,
                 noise: float = 0.3, scale_sigma: float = 1.0, per_coord_scale: bool = False,
                 tensors=None, boost: float = 1.0, boost_frac: float = 0.0, corr: float = 0.7):
        if grad_dtype not in ("f32", "bf16"):
            raise ValueError(grad_dtype)
        self.d, self.N, self.seed, self.grad_dtype = int(d), int(N), int(seed), grad_dtype
        if per_coord_scale:
            z = normals(seed, STREAM_SCALE_COORD, d).astype(np.float64)
            self.scale = np.exp(scale_sigma * z).astype(np.float32)
            self.seg_begin = np.zeros(1, dtype=np.int64)
        else:
            sizes = list(tensors) if tensors else [d]
            if sum(sizes) != d:
                raise ValueError("tensor sizes must add up to d")
            z = normals(seed, STREAM_SCALE_TENSOR, len(sizes)).astype(np.float64)
            self.scale = np.exp(scale_sigma * z).astype(np.float32)
            self.seg_begin = np.concatenate([[0], np.cumsum(sizes)[:-1]]).astype(np.int64)
        self.plan = _Plan(
            family=family, out_bf16=1 if grad_dtype == "bf16" else 0, d=self.d, N=self.N,
            per_coord=1 if per_coord_scale else 0, seed=self.seed, noise=noise,
            c_shared=float(np.float32(np.sqrt(corr))), c_own=float(np.float32(np.sqrt(1 - corr))),
            boost=boost, boost_threshold=int(round(boost_frac * 2.0 ** 32)),
            nseg=int(self.seg_begin.size), seg_begin=self.seg_begin.ctypes.data,
            scale=self.scale.ctypes.data)
        self._dev_tables = None

    @classmethod
    def for_workload(cls, w: Workload, N: int | None = None, d: int | None = None):
        return cls(d or w.d, N or w.N, w.data_seed, grad_dtype=w.grad_dtype, family=w.family,
                   noise=w.noise, scale_sigma=w.scale_sigma, per_coord_scale=w.per_coord_scale,
                   tensors=w.tensors if d is None else None, boost=w.boost,
                   boost_frac=w.boost_frac, corr=w.corr)

    @property
    def np_dtype(self):
        return np.uint16 if self.grad_dtype == "bf16" else np.float32

    def fill_host(self, t: int, i0: int = 0, i1: int | None = None, j0: int = 0,
                  j1: int | None = None) -> np.ndarray:
        """Gradients of workers [i0, i1) at coordinates [j0, j1) for step t
        (float32, or uint16 bf16 bit patterns)."""
        i1 = self.N if i1 is None else i1
        j1 = self.d if j1 is None else j1
        out = np.empty((i1 - i0, j1 - j0), dtype=self.np_dtype)
        rc = _host_lib().synth_fill_host(ctypes.byref(self.plan), t, i0, i1, j0, j1,
                                         out.ctypes.data, j1 - j0)
        if rc != 0:
            raise ValueError("synth_fill_host: bad range")
        return out

    def fill_device(self, t: int, out, stream=None) -> None:
        """Fill a device tensor holding N*d gradients for step t."""
        import torch
        if out.numel() != self.N * self.d or out.element_size() != np.dtype(self.np_dtype).itemsize:
            raise ValueError("output tensor has the wrong size or dtype")
        if not out.is_contiguous():
            raise ValueError("output tensor must be contiguous")
        if self._dev_tables is None or self._dev_tables[0].device != out.device:
            self._dev_tables = (torch.from_numpy(self.seg_begin).to(out.device),
                                torch.from_numpy(self.scale).to(out.device))
        plan = _Plan.from_buffer_copy(self.plan)
        plan.seg_begin = self._dev_tables[0].data_ptr()
        plan.scale = self._dev_tables[1].data_ptr()
        s = stream if stream is not None else torch.cuda.current_stream(out.device)
        rc = _dev_lib().synth_fill_device(ctypes.byref(plan), t, out.data_ptr(), s.cuda_stream)
        if rc != 0:
            raise RuntimeError(f"synth_fill_device failed: hip error {rc}")
