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
    from oracle import build as ob
    if not os.path.exists(ob.LIB):
        ob.build_oracle()
    try:
        from synth import build as sb
    except ImportError:
        return
    if not os.path.exists(sb.HOST_LIB):
        sb.build_synth_host()


_ensure_built()
