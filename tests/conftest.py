"""Shared pytest set-up: the `gpu` marker and on-demand builds of missing libraries."""
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs through the HIP path)")


def _ensure_built():
    # Load what is built; build only what is missing (a fresh checkout).
    import torch  # noqa: F401  (first: the process then holds torch's HIP runtime)
    import __graft_entry__ as ge
    ob = ge._load_by_path("_arc_oracle_build", "oracle/build.py")
    if not os.path.exists(ob.LIB):
        ob.build_oracle()
    sb = ge._load_by_path("_arc_synth_build", "synth/build.py")
    if not os.path.exists(sb.HOST_LIB):
        sb.build_synth_host()
    if not os.path.exists(sb.DEV_LIB):
        sb.build_synth_dev()
    lb = ge._load_by_path("_arc_lib_build", "paper_2510_26709_amd/build.py")
    if not os.path.exists(lb.LIB):
        lb.build_lib()


_ensure_built()
