"""The C ABI of libarctopk on the CPU: the library loads, exports every entry
point the header declares, its struct layout matches the binding, and invalid
arguments are rejected before any device work (no GPU needed)."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2510_26709_amd as arc
from paper_2510_26709_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "libarctopk.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(arc_[a-z_]+)\s*\(", text)))


def test_header_declares_the_documented_entry_points():
    names = declared_functions()
    for must in ("arc_create", "arc_step", "arc_destroy"):
        assert must in names
    assert set(names) == set(arc.EXPORTED)


def test_library_exports_every_declared_symbol():
    out = subprocess.run(["nm", "-D", "--defined-only", arc.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = {ln.split()[-1] for ln in out.splitlines() if " T " in ln}
    for name in declared_functions():
        assert name in exported, name
        assert getattr(_lib._lib, name) is not None


def test_config_layout_matches_header(tmp_path):
    src = tmp_path / "layout.c"
    src.write_text(
        '#include <stddef.h>\n#include <stdio.h>\n#include "libarctopk.h"\n'
        "int main(void){printf(\"%zu\", sizeof(arc_config));"
        + "".join(f'printf(" %zu", offsetof(arc_config, {f}));'
                  for f, _ in _lib.arc_config._fields_)
        + "return 0;}\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)],
                   check=True)
    vals = [int(x) for x in subprocess.run([str(exe)], capture_output=True, text=True,
                                           check=True).stdout.split()]
    assert vals[0] == ctypes.sizeof(_lib.arc_config)
    for (f, _), off in zip(_lib.arc_config._fields_, vals[1:]):
        assert getattr(_lib.arc_config, f).offset == off, f


BASE = dict(d=4096, N=2, n=64, r=4, K=3, eta=0.1, seed=1)


@pytest.mark.parametrize("override", [
    dict(d=0), dict(d=-5), dict(n=0), dict(N=0), dict(N=70000), dict(r=0), dict(r=33),
    dict(K=-1), dict(eta=-0.01), dict(eta=1.5), dict(eta=float("nan")),
    dict(grad_dtype=7), dict(reserved=1), dict(d=(2**31) * 3, n=1),
    dict(buckets=([0, 10, 63], [1, 1])),        # does not end at m = 64
    dict(buckets=([1, 10, 64], [1, 1])),        # does not start at 0
    dict(buckets=([0, 10, 10, 64], [1, 1, 1])),  # empty bucket
    dict(buckets=([0, 10, 64], [1, -2])),       # negative K
])
def test_create_rejects_invalid_config(override):
    kw = dict(BASE, **override)
    cfg, keep = arc.make_config(**kw)
    out = ctypes.c_void_p(12345)
    st = _lib._lib.arc_create(ctypes.byref(cfg), None, ctypes.byref(out))
    assert st == arc.ARC_ERR_INVALID
    assert out.value is None
    assert arc.arc_last_error() != ""


def test_create_rejects_null_arguments():
    cfg, _ = arc.make_config(**BASE)
    assert _lib._lib.arc_create(None, None, ctypes.byref(ctypes.c_void_p())) == arc.ARC_ERR_INVALID
    assert _lib._lib.arc_create(ctypes.byref(cfg), None, None) == arc.ARC_ERR_INVALID
    cfg.num_buckets = 2  # arrays still NULL
    assert _lib._lib.arc_create(ctypes.byref(cfg), None,
                                ctypes.byref(ctypes.c_void_p())) == arc.ARC_ERR_INVALID


def test_null_context_paths():
    L = _lib._lib
    assert L.arc_destroy(None) == arc.ARC_OK
    assert L.arc_num_rows(None) == -1
    assert L.arc_selected_rows(None) == -1
    assert L.arc_step(None, 0, 1, 2, 3, 4, 5) == arc.ARC_ERR_INVALID
    for fn in ("arc_debug_sigma", "arc_debug_sketch", "arc_set_projection"):
        assert getattr(L, fn)(None, None) == arc.ARC_ERR_INVALID
    assert L.arc_timing_enable(None, 1) == arc.ARC_ERR_INVALID
    assert L.arc_debug_projection(None, 0, None) == arc.ARC_ERR_INVALID
    assert L.arc_describe(None, None, 0) == arc.ARC_ERR_INVALID
    assert L.arc_timing_read(None, None, None) == arc.ARC_ERR_INVALID


def test_status_strings():
    for code, name in [(0, "ARC_OK"), (1, "ARC_ERR_INVALID"), (2, "ARC_ERR_NOMEM"),
                       (3, "ARC_ERR_DEVICE"), (4, "ARC_ERR_UNSUPPORTED")]:
        assert arc.arc_status_str(code) == name
    assert arc.arc_status_str(99) == "ARC_ERR_UNKNOWN"


def test_binding_raises_with_reason():
    cfg, _ = arc.make_config(**dict(BASE, r=0))
    with pytest.raises(arc.ArcError, match="r must be"):
        arc.arc_create(cfg)


def test_tensor_layout_matches_header(tmp_path):
    src = tmp_path / "tlayout.c"
    src.write_text(
        '#include <stddef.h>\n#include <stdio.h>\n#include "libarctopk.h"\n'
        'int main(void){printf("%zu %zu %zu %zu", sizeof(arc_tensor),'
        " offsetof(arc_tensor, rows), offsetof(arc_tensor, cols),"
        " offsetof(arc_tensor, K));return 0;}\n")
    exe = tmp_path / "tlayout"
    subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)],
                   check=True)
    vals = [int(x) for x in subprocess.run([str(exe)], capture_output=True, text=True,
                                           check=True).stdout.split()]
    assert vals == [ctypes.sizeof(_lib.arc_tensor), _lib.arc_tensor.rows.offset,
                    _lib.arc_tensor.cols.offset, _lib.arc_tensor.K.offset]


TBASE = dict(d=64 * 96 + 300, N=2, r=4, eta=0.1, seed=1,
             tensors=[(64, 96, 5), (1, 300, 1)])


@pytest.mark.parametrize("override", [
    dict(tensors=[(64, 96, 5), (1, 299, 1)]),      # covers d - 1
    dict(tensors=[(64, 96, 5), (1, 301, 1)]),      # covers d + 1
    dict(tensors=[(0, 96, 5), (1, 6444, 1)]),      # empty tensor
    dict(tensors=[(64, 0, 5), (1, 6444, 1)]),      # zero width
    dict(tensors=[(64, 96, -1), (1, 300, 1)]),     # negative K
    dict(n=96),                                    # n with tensors
    dict(K=3),                                     # global K with tensors
    dict(buckets=([0, 65], [1])),                  # buckets with tensors
    dict(compressor=3),
    dict(tensors=[(2**40, 2**40, 1)], d=2**40),   # rows*cols would overflow int64
])
def test_create_rejects_invalid_tensor_config(override):
    kw = dict(TBASE, **override)
    cfg, keep = arc.make_config(**kw)
    out = ctypes.c_void_p(12345)
    st = _lib._lib.arc_create(ctypes.byref(cfg), None, ctypes.byref(out))
    assert st == arc.ARC_ERR_INVALID, arc.arc_last_error()
    assert out.value is None


def test_create_rejects_null_tensor_array():
    cfg, keep = arc.make_config(**TBASE)
    cfg.tensors = None
    assert _lib._lib.arc_create(ctypes.byref(cfg), None,
                                ctypes.byref(ctypes.c_void_p())) == arc.ARC_ERR_INVALID
    assert "tensors" in arc.arc_last_error()


def test_payload_elems_of_null_context():
    assert _lib._lib.arc_payload_elems(None) == -1


def test_library_projection_matches_oracle_bitwise_on_host():
    """arc_projection is host code in the library; the oracle generates V from
    its own SplitMix64 and Box-Muller code.  No device is touched."""
    import numpy as np

    import oracle
    for seed, t, n, r in ((2003, 0, 768, 4), (7, 19, 147, 3), (2**64 - 1, 123456, 33, 1),
                          (0, 5, 1, 32)):
        got = np.empty((n, r), np.float32)
        arc.arc_projection(seed, t, n, r, got)
        want = oracle.projection(seed, t, n, r)
        assert got.tobytes() == want.tobytes(), (seed, t, n, r)


@pytest.mark.parametrize("args", [(1, -1, 4, 4), (1, 0, 0, 4), (1, 0, 4, 0), (1, 0, 4, 33)])
def test_projection_rejects_bad_arguments(args):
    import numpy as np
    buf = np.empty(64, np.float32)
    with pytest.raises(arc.ArcError):
        arc.arc_projection(*args, buf)
    assert _lib._lib.arc_projection(1, 0, 4, 4, None) == arc.ARC_ERR_INVALID


def test_model_config_layout_matches_header(tmp_path):
    src = tmp_path / "mlayout.c"
    fields = [f for f, _ in _lib.arc_model_config._fields_]
    src.write_text(
        '#include <stddef.h>\n#include <stdio.h>\n#include "libarctopk.h"\n'
        'int main(void){printf("%zu", sizeof(arc_model_config));'
        + "".join(f'printf(" %zu", offsetof(arc_model_config, {f}));' for f in fields)
        + "return 0;}\n")
    exe = tmp_path / "mlayout"
    subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)],
                   check=True)
    vals = [int(x) for x in subprocess.run([str(exe)], capture_output=True, text=True,
                                           check=True).stdout.split()]
    assert vals[0] == ctypes.sizeof(_lib.arc_model_config)
    for f, off in zip(fields, vals[1:]):
        assert getattr(_lib.arc_model_config, f).offset == off, f


def test_model_step_rejects_null_context_and_config():
    L = _lib._lib
    mc = arc.make_model_config("sgd", lr=0.1)
    assert L.arc_model_step(None, ctypes.byref(mc), 0, 1, 2, 3, 4, 5, None, None, 6, 7) == \
        arc.ARC_ERR_INVALID
    assert L.arc_model_step(12345, None, 0, 1, 2, 3, 4, 5, None, None, 6, 7) == \
        arc.ARC_ERR_INVALID


def test_static_step_rejects_before_any_device_work():
    """arc_step_static checks the configuration and sizes its static device
    scratch on the host: an invalid configuration, and one whose buffers
    exceed ARC_STATIC_SCRATCH_BYTES, are rejected with no HIP call (this runs
    without a GPU)."""
    L = _lib._lib
    assert L.arc_step_static(None, None, 0, 1, 2, 3, 4, 5) == arc.ARC_ERR_INVALID
    cfg, keep = arc.make_config(**dict(BASE, r=0))
    assert L.arc_step_static(ctypes.byref(cfg), None, 0, 1, 2, 3, 4, 5) == arc.ARC_ERR_INVALID
    # 2^24 rows of 4 values, r = 4: a 256 MiB per-worker sketch
    cfg, keep = arc.make_config(d=1 << 26, N=1, n=4, r=4, K=1, eta=0.1, seed=1)
    assert L.arc_step_static(ctypes.byref(cfg), None, 0, 1, 2, 3, 4, 5) == arc.ARC_ERR_INVALID
    msg = arc.arc_last_error()
    assert "static" in msg and str(arc.ARC_STATIC_SCRATCH_BYTES) in msg, msg
    with pytest.raises(arc.ArcError, match="static"):
        arc.arc_step_static(cfg, None, 0, 1, 2, 3, 4, 5)
